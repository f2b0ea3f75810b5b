"""The C ABI library loads, exports every symbol its header declares, and
validates host-side arguments before touching the GPU (no GPU needed)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "nebulasd.h")


@pytest.fixture(scope="module")
def lib():
    import paper_2609_29364_amd as nsd
    if not os.path.exists(nsd.LIB_PATH):
        from paper_2609_29364_amd.build import build
        build()
    return nsd.lib()


def declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(nsd_\w+)\s*\(", src)))


def test_header_declares_the_round(lib):
    names = declared()
    assert {"nsd_kv_gather", "nsd_verify_attention", "nsd_spec_accept",
            "nsd_verify_attention_workspace_size", "nsd_last_error", "nsd_version"} <= set(names)


def test_every_declared_symbol_is_exported(lib):
    for name in declared():
        assert hasattr(lib, name), name


def test_version_and_error_string(lib):
    assert lib.nsd_version() >= 1
    assert isinstance(lib.nsd_last_error(), bytes)


def test_gather_validation(lib):
    # bad head_dim, bad block size, bad layer range, NULLs: rejected before any HIP call
    st = lib.nsd_kv_gather(None, None, 4, None, None, 4, None, None, 3, 1, 0, 1, 2, 16, 96, None)
    assert st == 3 and b"head_dim" in lib.nsd_last_error()
    assert lib.nsd_kv_gather(None, None, 4, None, None, 4, None, None, 3, 1, 0, 1, 2, 8, 64, None) == 3
    assert lib.nsd_kv_gather(None, None, 4, None, None, 4, None, None, 3, 2, 1, 2, 2, 16, 64, None) == 2
    assert lib.nsd_kv_gather(None, None, 4, None, None, 4, None, None, 3, 1, 0, 1, 2, 16, 64, None) == 1
    assert lib.nsd_kv_gather(None, None, 4, None, None, 4, None, None, -1, 1, 0, 1, 2, 16, 64, None) == 2
    # empty plan is a no-op even with NULL pointers
    assert lib.nsd_kv_gather(None, None, 4, None, None, 4, None, None, 0, 1, 0, 1, 2, 16, 64, None) == 0


def test_attention_validation(lib):
    f = lib.nsd_verify_attention
    args = lambda **kw: [kw.get(k, v) for k, v in [
        ("q", None), ("k", None), ("v", None), ("nb", 64), ("bt", None), ("mbps", 16),
        ("sl", None), ("qi", None), ("bs", 4), ("hq", 4), ("hkv", 2), ("d", 64), ("blk", 16),
        ("mq", 5), ("msl", 256), ("scale", 0.125), ("out", None), ("ws", None), ("wsb", 0),
        ("stream", None)]]
    assert f(*args(d=80)) == 3
    assert f(*args(hq=5)) == 2
    assert f(*args(blk=32)) == 3
    assert f(*args(mq=40)) == 3                      # (4/2)*40 rows > 64
    assert f(*args(scale=float("nan"))) == 2
    assert f(*args(bs=0)) == 0                       # no-op
    assert f(*args()) == 1                           # NULL pointers
    assert b"NULL" in lib.nsd_last_error()
    size = lib.nsd_verify_attention_workspace_size
    assert size(4, 4, 2, 64, 5, 256) >= 0
    assert size(4, 5, 2, 64, 5, 256) == 0            # invalid sizes -> 0
    big = size(256, 32, 8, 128, 5, 4096)
    assert big > 0 and big % 16 == 0
    # a row count past 2^31 is refused, not wrapped
    assert f(*args(hq=2**30, hkv=1, mq=2**30)) == 3
    assert size(4, 2**30, 1, 64, 2**30, 256) == 0
    assert size(4, 2**31 - 1, 1, 64, 128, 256) == 0


def test_layer_range_overflow_is_refused(lib):
    # layer0 + n_layers past 2^31 - 1 is a shape error, found without wrapping
    st = lib.nsd_kv_gather(None, None, 4, None, None, 4, None, None, 3, 8, 7, 2**31 - 1, 2, 16,
                           64, None)
    assert st == 2 and b"layer range" in lib.nsd_last_error()


def test_attention_workspace_check(lib):
    need = lib.nsd_verify_attention_workspace_size(256, 32, 8, 128, 5, 4096)
    fake = ctypes.c_void_p(16)  # never dereferenced: the size check fails first
    st = lib.nsd_verify_attention(fake, fake, fake, 100, fake, 256, fake, fake, 256, 32, 8, 128,
                                  16, 5, 4096, 0.08, fake, fake, need - 16, None)
    assert st == 4 and b"workspace" in lib.nsd_last_error()


def test_accept_validation(lib):
    f = lib.nsd_spec_accept
    z = (None, 0, None)
    assert f(None, None, None, None, None, 4, 1001, 4, None, None, *z) == 3   # vocab % 4
    assert f(None, None, None, None, None, 4, 1 << 20, 4, None, None, *z) == 3
    assert f(None, None, None, None, None, 4, 1000, 64, None, None, *z) == 3
    assert f(None, None, None, None, None, 1 << 30, 1000, 4, None, None, *z) == 2
    assert f(None, None, None, None, None, 0, 1000, 4, None, None, *z) == 0
    assert f(None, None, None, None, None, 4, 1000, 4, None, None, *z) == 1
    size = lib.nsd_spec_accept_workspace_size
    assert size(256, 151936) == ((256 * 594 * 8 + 255) // 256) * 256 + 256 * 4
    assert size(-1, 1000) == 0
    # rows and probabilities present, workspace too small: refused before any launch
    fake = 1 << 20
    st = f(fake, fake, fake, fake, fake, 4, 1000, 4, fake, fake, fake, 16, None)
    assert st == 4 and b"workspace" in lib.nsd_last_error()


def test_sample_validation(lib):
    f = lib.nsd_sample
    z = (None, 0, None)
    assert f(None, 1000, None, 4, 1001, None, 1, *z) == 3                # vocab % 4
    assert f(None, 996, None, 4, 1000, None, 1, *z) == 2                 # row_stride < vocab
    assert f(None, 1002, None, 4, 1000, None, 1, *z) == 2                # row_stride % 4
    assert f(None, 1000, None, 4, 1000, None, 0, *z) == 2                # out_stride
    assert f(None, 1000, None, -1, 1000, None, 1, *z) == 2
    assert f(None, 1000, None, 0, 1000, None, 1, *z) == 0
    assert f(None, 1000, None, 4, 1000, None, 1, *z) == 1
    assert f(8, 1000, 8, 4, 1000, 8, 1, *z) == 2 and b"aligned" in lib.nsd_last_error()
    assert f(16, 1000, 16, 4, 1000, 16, 1, *z) == 4                      # no workspace


def test_copy_plan_validation(lib):
    f = lib.nsd_copy_plan
    plan = (ctypes.c_int64 * 6)(0, 0, 64, 64, 64, 64)
    fake = ctypes.c_void_p(16)  # never dereferenced: every case fails before any copy
    assert f(fake, 128, fake, 128, plan, 2, 1 << 20, 3, None) == 2          # bad direction
    assert f(fake, 128, fake, 128, plan, 2, 0, 1, None) == 2                # chunk < 1
    assert f(fake, 128, fake, 128, plan, -1, 1 << 20, 1, None) == 2         # n < 0
    assert f(None, 128, None, 128, None, 0, 1 << 20, 1, None) == 0          # empty plan
    assert f(None, 128, fake, 128, plan, 2, 1 << 20, 1, None) == 1          # NULL
    assert f(fake, 100, fake, 128, plan, 2, 1 << 20, 1, None) == 2          # src overrun
    assert b"leaves its buffers" in lib.nsd_last_error()
    bad = (ctypes.c_int64 * 3)(0, -8, 8)
    assert f(fake, 128, fake, 128, bad, 1, 1 << 20, 2, None) == 2          # negative offset


def test_append_commit_alias_validation(lib):
    f = lib.nsd_kv_append
    fake = ctypes.c_void_p(16)
    assert f(fake, fake, 8, fake, fake, fake, 4, fake, fake, 2, 8, 2, 8, 64, None) == 3    # block size
    assert f(fake, fake, 8, fake, fake, fake, 4, fake, fake, 2, 8, 2, 16, 96, None) == 3   # head_dim
    assert f(fake, fake, 8, fake, fake, fake, 0, fake, fake, 2, 8, 2, 16, 64, None) == 2   # no blocks
    assert f(None, None, 8, None, None, None, 4, None, None, 0, 8, 2, 16, 64, None) == 0   # bs == 0
    assert f(None, fake, 8, fake, fake, fake, 4, fake, fake, 2, 8, 2, 16, 64, None) == 1   # NULL
    odd = ctypes.c_void_p(24)   # never dereferenced: refused before any launch
    assert f(odd, fake, 8, fake, fake, fake, 4, fake, fake, 2, 8, 2, 16, 64, None) == 2    # alignment
    assert b"16-byte aligned" in lib.nsd_last_error()
    g = lib.nsd_commit_lengths
    assert g(None, None, None, None, 0, None) == 0
    assert g(None, None, None, None, -1, None) == 2
    assert g(fake, None, fake, fake, 3, None) == 1
    out = ctypes.c_void_p()
    assert lib.nsd_host_alias(None, ctypes.byref(out)) == 1


def test_probe_library_exports_and_validates():
    """The bandwidth-probe library (measurement only) exports what its header
    declares and refuses bad arguments before any launch."""
    from paper_2609_29364_amd.build import PROBE_LIB_PATH, build
    if not os.path.exists(PROBE_LIB_PATH):
        build()
    plib = ctypes.CDLL(PROBE_LIB_PATH)
    src = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "nsd_probe.h")).read(),
                 flags=re.S)
    names = sorted(set(re.findall(r"\b(nsd_\w+)\s*\(", src)))
    assert names == ["nsd_probe_tiles", "nsd_probe_tiles_writer"]
    for name in names:
        assert hasattr(plib, name), name
    f = plib.nsd_probe_tiles
    f.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                  ctypes.c_void_p, ctypes.c_void_p]
    fake = 16   # never dereferenced: every case fails before any launch
    assert f(None, 8, None, 0, fake, None, 4, 1, fake, None) == 1        # no source
    assert f(fake, 8, None, 8, fake, fake, 4, 1, fake, None) == 1        # writes without dst
    assert f(fake, 8, None, 0, fake, None, 6, 1, fake, None) == 2        # waves % 4
    assert f(fake, 0, None, 0, fake, None, 4, 1, fake, None) == 2        # empty source
    assert f(fake, 8, None, 0, fake, None, 4, -1, fake, None) == 2       # steps < 0
    w = plib.nsd_probe_tiles_writer
    w.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                  ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    assert w(fake, 8, None, 8, fake, fake, 1, 4, 1, fake, None) == 1     # no destination
    assert w(fake, 8, fake, 8, fake, None, 1, 4, 1, fake, None) == 1     # no write list
    assert w(None, 8, fake, 8, None, fake, 1, 4, 1, fake, None) == 1     # reads without source
    assert w(fake, 8, fake, 8, fake, fake, 1, 6, 1, fake, None) == 2     # waves % 4
    assert w(fake, 8, fake, 0, fake, fake, 1, 4, 1, fake, None) == 2     # empty destination
    assert w(fake, 8, fake, 8, fake, fake, -1, 4, 1, fake, None) == 2    # write_per < 0
    assert w(fake, 8, fake, 8, fake, fake, 1, 4, -1, fake, None) == 2    # steps < 0


def test_attention_wave_hook(lib):
    # the explicit wave-count hook replaces the device's count for the workspace query
    import paper_2609_29364_amd as nsd
    assert lib.nsd_attention_waves() == 0
    assert lib.nsd_set_attention_waves(6) == 2 and lib.nsd_set_attention_waves(-4) == 2
    assert lib.nsd_attention_waves() == 0
    small = big = None
    with nsd.attention_waves(8):
        assert lib.nsd_attention_waves() == 8
        small = lib.nsd_verify_attention_workspace_size(4, 4, 2, 64, 5, 256)
        with nsd.attention_waves(64):
            big = lib.nsd_verify_attention_workspace_size(4, 4, 2, 64, 5, 256)
        assert lib.nsd_attention_waves() == 8
    assert lib.nsd_attention_waves() == 0
    assert 0 < small < big


def _plan(cfg_name="tiny", **kw):
    from workload import CONFIGS, custom_config, make_meta
    cfg = custom_config(**kw) if kw else CONFIGS[cfg_name]
    return make_meta(cfg)


def _check(meta, **over):
    import paper_2609_29364_amd as nsd
    args = dict(block_table=meta.block_table, seq_lens=meta.seq_lens, q_indptr=meta.q_indptr,
                num_blocks=meta.num_blocks, max_q_per_seq=meta.max_q,
                max_seq_len=meta.max_seq_len, stage_table=meta.stage_table,
                stage_num_blocks=meta.stage_num_blocks, total_q=meta.total_q)
    args.update(over)
    nsd.check_plan(**args)


def test_check_plan_accepts_the_workloads(lib):
    from workload import CONFIGS, make_meta
    for name in CONFIGS:
        meta = make_meta(CONFIGS[name])
        _check(meta)                     # fused plan (stage table)
        _check(meta, stage_table=None)   # plain attention plan


def test_check_plan_rejects_each_violation(lib):
    import numpy as np
    import paper_2609_29364_amd as nsd
    meta = _plan(seed=61, bs=6, k_lo=1, k_hi=5, n_arriving=3, pool_blocks=None)
    cases = []
    qi = meta.q_indptr.copy(); qi[0] = 1; cases.append(("q_indptr[0]", dict(q_indptr=qi)))
    cases.append(("q has", dict(total_q=meta.total_q + 1)))
    qi = meta.q_indptr.copy(); qi[2] = qi[1]; cases.append(("query rows", dict(q_indptr=qi)))
    qi = meta.q_indptr.copy(); qi[3] = qi[2] - 1; cases.append(("query rows", dict(q_indptr=qi)))
    cases.append(("query rows", dict(max_q_per_seq=int(np.diff(meta.q_indptr).max()) - 1)))
    sl = meta.seq_lens.copy(); sl[1] = 0; cases.append(("seq_len", dict(seq_lens=sl)))
    cases.append(("seq_len", dict(max_seq_len=int(meta.seq_lens.max()) - 1)))
    bt = meta.block_table.copy(); bt[2, 0] = meta.num_blocks; cases.append(("pool id", dict(block_table=bt)))
    bt = meta.block_table.copy(); bt[2, 0] = -1; cases.append(("pool id", dict(block_table=bt)))
    bt = meta.block_table.copy(); bt[3, 0] = bt[4, 0]; cases.append(("used twice", dict(block_table=bt)))
    arr = int(np.nonzero(meta.arriving)[0][0])
    st = meta.stage_table.copy(); st[arr, 1] = meta.stage_num_blocks
    cases.append(("staging id", dict(stage_table=st)))
    others = np.nonzero(meta.arriving)[0]
    st = meta.stage_table.copy(); st[others[1], 0] = st[others[0], 0]
    cases.append(("staging block", dict(stage_table=st)))
    for needle, over in cases:
        with pytest.raises(nsd.NsdError) as e:
            _check(meta, **over)
        assert needle in str(e.value), (needle, str(e.value))
    # a plain attention plan may share a pool block between requests (read only)
    bt = meta.block_table.copy(); bt[3, 0] = bt[4, 0]
    _check(meta, block_table=bt, stage_table=None)
    # entries past a request's blocks are not checked
    bt = meta.block_table.copy()
    n0 = -(-int(meta.seq_lens[0]) // 16)
    if n0 < bt.shape[1]:
        bt[0, n0:] = -7
        _check(meta, block_table=bt)


def test_check_pairs(lib):
    import numpy as np
    import paper_2609_29364_amd as nsd
    meta = _plan()
    nsd.check_pairs(meta.src_ids, meta.dst_ids, meta.stage_num_blocks, meta.num_blocks)
    nsd.check_pairs(np.zeros(0, np.int32), np.zeros(0, np.int32), 0, 0)
    for needle, s, d in [("source id", [0, 9], [1, 2]), ("destination id", [0, 1], [1, 64]),
                         ("named twice", [0, 1], [3, 3]), ("source id", [-1], [0])]:
        with pytest.raises(nsd.NsdError) as e:
            nsd.check_pairs(np.array(s), np.array(d), 9, 64)
        assert needle in str(e.value)


def test_windowed_copy_and_plan_validation(lib):
    import numpy as np
    f = lib.nsd_copy_plan_windowed
    plan = (ctypes.c_int64 * 3)(0, 0, 64)
    fake = ctypes.c_void_p(16)  # never dereferenced: every case fails before any copy
    assert f(fake, 128, fake, 128, plan, 1, 1 << 20, 0, 1, None) == 2       # window < 1
    assert f(fake, 128, fake, 128, plan, 1, 0, 1 << 20, 1, None) == 2       # chunk < 1
    assert f(None, 0, None, 0, None, 0, 1 << 20, 1 << 20, 1, None) == 0     # empty plan
    # h2d plan: capacity too small reports the length needed
    n = ctypes.c_int64()
    ext = np.array([0, 10], np.int64)
    st = np.array([[3, 4, -1], [5, 6, 7]], np.int32)
    arr = np.array([1, 1], np.uint8)
    sl = np.array([20, 40], np.int32)
    out = np.zeros((8, 3), np.int64)
    h = lib.nsd_h2d_plan
    assert h(ext.ctypes.data, st.ctypes.data, 3, arr.ctypes.data, sl.ctypes.data, 2, 100,
             out.ctypes.data, 2, ctypes.byref(n)) == 4 and n.value == 5
    assert h(ext.ctypes.data, st.ctypes.data, 3, arr.ctypes.data, sl.ctypes.data, 2, 100,
             out.ctypes.data, 8, ctypes.byref(n)) == 0 and n.value == 5
    assert out[:5].tolist() == [[0, 300, 100], [100, 400, 100], [1000, 500, 100],
                                [1100, 600, 100], [1200, 700, 100]]
    sl2 = np.array([20, 49], np.int32)       # 4 blocks in a 3-entry table
    assert h(ext.ctypes.data, st.ctypes.data, 3, arr.ctypes.data, sl2.ctypes.data, 2, 100,
             out.ctypes.data, 8, ctypes.byref(n)) == 2
    w = lib.nsd_writeback_pairs
    bt = np.array([[9, 8, 7], [6, 5, 4]], np.int32)
    s_ = np.zeros(8, np.int32)
    d_ = np.zeros(8, np.int32)
    hl = np.array([15, 16], np.int32)
    nl = np.array([17, 33], np.int32)
    assert w(bt.ctypes.data, 3, ext.ctypes.data, hl.ctypes.data, nl.ctypes.data, 2,
             s_.ctypes.data, d_.ctypes.data, 8, ctypes.byref(n)) == 0 and n.value == 4
    assert s_[:4].tolist() == [9, 8, 5, 4] and d_[:4].tolist() == [0, 1, 11, 12]
    nl_bad = np.array([17, 49], np.int32)    # past the table
    assert w(bt.ctypes.data, 3, ext.ctypes.data, hl.ctypes.data, nl_bad.ctypes.data, 2,
             s_.ctypes.data, d_.ctypes.data, 8, ctypes.byref(n)) == 2
    assert w(bt.ctypes.data, 3, ext.ctypes.data, hl.ctypes.data, nl.ctypes.data, 2,
             s_.ctypes.data, d_.ctypes.data, 1, ctypes.byref(n)) == 4 and n.value == 4
