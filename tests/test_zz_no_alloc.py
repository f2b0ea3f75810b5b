"""The acceptance entry point that allocates nothing (its scratch is a static
device array per GPU), called through the C ABI, against nsd_spec_accept with
a caller workspace: bit-identical accepted lengths and tokens on consecutive
calls, the second smaller than the first (the scratch keeps the previous
call's contents), and on a batch that takes the one-pass kernel; the size
limit is refused."""
import numpy as np
import pytest
import torch

import paper_2609_29364_amd as nsd
from workload import custom_config, make_meta, make_accept
from parity import i32, check_accept

pytestmark = pytest.mark.gpu


def _inputs(seed, bs, vocab, device):
    cfg = custom_config(seed=seed, bs=bs, k_lo=0, k_hi=6, ctx_lo=8, ctx_hi=40, vocab=vocab,
                        n_arriving=0, pool_blocks=None)
    meta = make_meta(cfg)
    return meta, make_accept(cfg, meta, device)


def _both(meta, a, device):
    qi = i32(meta.q_indptr, device)
    k = int(meta.depth.max())
    ref_acc, ref_tok = nsd.spec_accept(a.p_target, a.q_draft, a.draft_tokens, a.uniforms, qi, k)
    acc = torch.full((meta.bs,), -5, dtype=torch.int32, device=device)
    tok = torch.full((meta.total_q,), -5, dtype=torch.int32, device=device)
    nsd.spec_accept_static(a.p_target, a.q_draft, a.draft_tokens, a.uniforms, qi, k, acc, tok)
    torch.cuda.synchronize()
    return ref_acc.cpu().numpy(), ref_tok.cpu().numpy(), acc.cpu().numpy(), tok.cpu().numpy()


def test_static_scratch_matches_workspace_entry_point(device):
    # two calls in a row on the two-kernel path (rows below the CU count), the
    # second smaller; then a batch with a row per CU (the one-pass kernel)
    for seed, bs, vocab in [(81, 200, 151936), (82, 37, 16388), (83, 300, 1000)]:
        meta, a = _inputs(seed, bs, vocab, device)
        ref_acc, ref_tok, acc, tok = _both(meta, a, device)
        assert np.array_equal(acc, ref_acc), f"bs={bs}: accepted lengths differ"
        assert np.array_equal(tok, ref_tok), f"bs={bs}: tokens differ"
        check_accept(a.p_target.cpu().numpy(), a.q_draft.cpu().numpy(),
                     a.draft_tokens.cpu().numpy(), a.uniforms.cpu().numpy(), meta.q_indptr,
                     acc, tok)


def test_static_scratch_refuses_batches_beyond_its_size(device):
    cap = nsd.lib().nsd_spec_accept_static_max_bytes()
    vocab = 151936
    bs = 1
    while nsd.accept_workspace_size(bs, vocab) <= cap:
        bs *= 2
    meta, a = _inputs(84, bs, 1000, device)
    # a vocabulary whose rows need more scratch than the array holds: refused
    # before any launch (the rows are never read)
    st = nsd.lib().nsd_spec_accept_static(
        a.p_target.data_ptr(), a.q_draft.data_ptr(), a.draft_tokens.data_ptr(),
        a.uniforms.data_ptr(), i32(meta.q_indptr, device).data_ptr(), bs, vocab,
        int(meta.depth.max()), 16, 16, None)
    assert st == 4 and b"scratch" in nsd.lib().nsd_last_error()
