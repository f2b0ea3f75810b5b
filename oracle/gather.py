"""Oracle for KV-state preparation (the gather of arriving requests' blocks).

Prepare(B, w) of Algorithm 1 makes the KV state of every request admitted to a
worker's batch resident on that worker before Run.  The state of a request
that arrives from elsewhere sits in a stable per-request extent of blocks
(Appendix E.1, Eq. E.1) and the copy is driven by compact numeric descriptors
(Appendix E.3/E.4).  The block is the unit of the paged cache (Section 3).

Here a copy plan is a list of (source block id, destination block id) pairs;
for every pair and every listed layer, the whole block -- all KV heads, all 16
token slots, both the K plane and the V plane -- is copied.  Blocks that no
pair names keep their bytes.
"""
import numpy as np


def kv_gather(src_k, src_v, dst_k, dst_v, src_ids, dst_ids, layer0=0, n_layers=None):
    """Return the destination planes after the copy plan has run.

    src_k, src_v: [layers][src_blocks][...] arrays (any dtype; bytes copied).
    dst_k, dst_v: [layers][dst_blocks][...] arrays, left untouched (copies returned).
    src_ids, dst_ids: the plan, pair i copies src block src_ids[i] to dst block dst_ids[i].
    Layers layer0 .. layer0 + n_layers - 1 are copied (default: all layers).
    """
    if n_layers is None:
        n_layers = dst_k.shape[0] - layer0
    out_k = np.array(dst_k, copy=True)
    out_v = np.array(dst_v, copy=True)
    for i in range(len(src_ids)):
        s, d = int(src_ids[i]), int(dst_ids[i])
        for layer in range(layer0, layer0 + n_layers):
            out_k[layer, d] = src_k[layer, s]
            out_v[layer, d] = src_v[layer, s]
    return out_k, out_v
