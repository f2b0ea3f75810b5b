"""Random calls of the library's host code, run by test_host_sanitizers.py in a
child process whose library was built with AddressSanitizer and
UndefinedBehaviorSanitizer on its host side (the process halts on the first
report, so a clean exit means no report).

usage: python host_fuzz.py <library> <seed> <iterations>

Two parts: the host-only entry points (plan checks, H2D and write-back plans,
batch reconstruction, simulation) with valid and invalid host arrays through
the Python binding, every call returning or raising NsdError / ValueError; and
the device entry points and size queries with random scalars (extreme ones
included) and fake device pointers that host code must never read; with no
GPU present, a call that passes its checks stops at the launch."""
import ctypes
import math
import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import paper_2609_29364_amd as nsd  # noqa: E402

I32_MAX = 2**31 - 1


def _wild(rng, n, lo, hi):
    """Mostly in [lo, hi); now and then negative, past hi or at 2^31 - 1."""
    v = rng.integers(lo, max(hi, lo + 1), n).astype(np.int64)
    m = rng.random(n)
    v = np.where(m < 0.03, -rng.integers(1, 1000, n), v)
    v = np.where((m >= 0.03) & (m < 0.05), hi + rng.integers(0, 1000, n), v)
    return np.where((m >= 0.05) & (m < 0.06), np.int64(I32_MAX), v)


def _i32(a):
    return np.clip(a, -2**31, I32_MAX).astype(np.int32)


def fuzz_host_only(rng, n_iter):
    from paper_2609_29364_amd import hostkv, schedule

    def call(f, *a, **k):
        try:
            f(*a, **k)
        except (nsd.NsdError, ValueError):
            pass

    for it in range(n_iter):
        bs, mb, nblocks = int(rng.integers(0, 40)), int(rng.integers(1, 12)), int(rng.integers(0, 200))
        lens = _i32(_wild(rng, bs, 1, 16 * mb + 1))
        bt = _i32(_wild(rng, bs * mb, 0, nblocks)).reshape(bs, mb)
        st = _i32(_wild(rng, bs * mb, 0, nblocks)).reshape(bs, mb)
        qi = np.concatenate([[0], np.cumsum(rng.integers(0, 6, bs))]).astype(np.int64)
        if bs and rng.random() < 0.2:
            qi[rng.integers(0, bs + 1)] += int(rng.integers(-5, 5))
        call(nsd.check_plan, bt, lens, _i32(qi), nblocks, int(rng.integers(0, 8)),
             int(rng.integers(0, 400)), stage_table=st if rng.random() < 0.5 else None,
             stage_num_blocks=nblocks, total_q=int(rng.integers(-1, 300)))
        n = int(rng.integers(0, 50))
        call(nsd.check_pairs, _i32(_wild(rng, n, 0, nblocks)), _i32(_wild(rng, n, 0, nblocks)),
             nblocks, nblocks)
        extent = _wild(rng, bs, 0, 1000)
        call(hostkv.h2d_plan, extent, st, rng.random(bs) < 0.5, lens,
             int(rng.choice([0, 4096, 32768, -1, 2**40])))
        host_len = _i32(_wild(rng, bs, 0, 16 * mb))
        new_len = _i32(host_len.astype(np.int64) + rng.integers(-3, 40, bs))
        call(hostkv.writeback_pairs, bt, extent, host_len, new_len)
        nc = int(rng.integers(0, 60))
        e = rng.random(nc) * 10
        if nc and rng.random() < 0.1:
            e[rng.integers(0, nc)] = rng.choice([math.nan, math.inf, -1.0])
        call(schedule.reconstruct, _i32(_wild(rng, nc, 0, 1000)), e, rng.random(nc) * 5,
             blocks=_wild(rng, nc, 0, 50) if rng.random() < 0.5 else None,
             tokens=_wild(rng, nc, 0, 800) if rng.random() < 0.5 else None,
             a_hat=float(rng.random() * 3), block_cap=int(rng.integers(-1, 400)),
             token_cap=int(rng.integers(-1, 5000)), b_max=int(rng.integers(0, 70)),
             g=float(rng.random() * 2), delta=float(rng.random()))
        if it % 10 == 0:
            sizes = np.sort(rng.integers(1, 64, 5)).astype(float)
            phi = [sizes, 1.0 + sizes * 0.1, np.clip(sizes / 64, 0, 1)]
            call(schedule.simulate, int(rng.integers(0, 4)), int(rng.integers(0, 4)),
                 int(rng.integers(0, 60)), int(rng.integers(0, 5)), phi, phi,
                 int(rng.integers(0, 40)), int(rng.integers(0, 40)), float(rng.random()),
                 float(rng.random()), float(rng.random()), float(rng.random()),
                 (int(rng.integers(0, 4)), int(rng.integers(0, 4))),
                 t_stop=float(rng.random() * 50), trace=bool(rng.random() < 0.5))


def fuzz_entry_points(rng, n_iter):
    lib = nsd.lib()
    fns = ["nsd_kv_gather", "nsd_verify_attention_workspace_size", "nsd_verify_attention",
           "nsd_gather_verify_attention", "nsd_spec_accept_workspace_size", "nsd_spec_accept",
           "nsd_sample", "nsd_kv_append", "nsd_commit_lengths"]
    i32 = [0, 1, 2, 3, 4, 7, 8, 16, 63, 64, 128, 256, 1000, 4096, 65535, 151936, 1 << 19, 2**30,
           -1, -16, I32_MAX, -2**31]
    i64 = i32 + [2**33, 2**40, 2**62, 2**63 - 1, -2**63]
    fake = [0x7F0000000000 + 256 * k for k in range(1, 16)] + [0x7F0000000008, 0x7F0000000002]

    def arg(t):
        if t is ctypes.c_void_p:
            return None if rng.random() < 0.15 else int(rng.choice(fake))
        if t is ctypes.c_int32:
            return int(rng.choice(i32)) if rng.random() < 0.7 else int(rng.integers(-5, 300))
        if t in (ctypes.c_int64, ctypes.c_size_t):
            v = int(rng.choice(i64)) if rng.random() < 0.7 else int(rng.integers(-5, 1 << 30))
            return v if t is ctypes.c_int64 else v & (2**64 - 1)
        if t is ctypes.c_float:
            return float(rng.choice([0.0, 0.088, 1.0, -1.0, np.inf, np.nan, 1e30]))
        raise TypeError(t)

    for it in range(n_iter):
        f = getattr(lib, fns[it % len(fns)])
        f(*[arg(t) for t in f.argtypes])


if __name__ == "__main__":
    nsd.LIB_PATH = sys.argv[1]
    nsd._lib = None
    rng = np.random.default_rng(int(sys.argv[2]))
    n = int(sys.argv[3])
    fuzz_host_only(rng, n)
    import torch
    if torch.cuda.device_count() == 0:   # counting devices does not initialise one
        # only where no GPU could run a launch that passes its checks
        fuzz_entry_points(rng, 10 * n)
    print("host fuzz: clean", flush=True)
