"""Seeded random configurations for the parity sweep: every model and request
field drawn over its valid range (head_dim, heads, block and page sizes,
layers, several requests with partial blocks and unaligned first rows, zero,
small and large shifts, tag subsets, repair fractions, output dtypes, both
RoPE pairings, partial rotary dimensions, scaled frequency tables and both
cache layouts), sized so that the oracle finishes each in seconds."""
import dataclasses

import numpy as np

from paper_2609_26219_amd import workloads as wl

SWEEP_SIZE = 32
MAX_ELEMS = 1_500_000  # layers x suffix tokens x heads x head_dim, per case


def sweep_case(i: int) -> "wl.Case":
    r = np.random.default_rng([26219, 8, i])
    D = int(r.choice([16, 32, 48, 64, 80, 96, 128, 160, 192, 256, 512]))
    H = int(r.integers(1, min(12, 4096 // D) + 1))
    while True:
        B = int(r.choice([1, 2, 3, 4, 5, 7, 8, 12, 16, 24, 32, 48, 64]))
        if (B * H * D) % 32 == 0:
            break
    P = int(2 ** r.integers(0, 7))
    L = int(r.integers(1, 4))
    nreq = int(r.integers(1, 4))
    n = [int(r.integers(1, 300)) for _ in range(nreq)]
    while L * sum(n) * H * D > MAX_ELEMS:
        n = [max(1, x // 2) for x in n]
    deltas = [int(r.choice([0, r.integers(-64, 65), r.integers(-20000, 20001)])) for _ in range(nreq)]
    rho0s = [int(r.integers(0, 3 * P + 50)) for _ in range(nreq)]
    tag_set = tuple(int(t) for t in np.flatnonzero(r.random(4) < 0.6)) or (int(r.integers(0, 4)),)
    out = int(r.integers(0, 2))
    theta = float(r.choice([1e4, 5e5, 1e6]))
    case = wl.make_custom(1000 + i, L=L, H=H, D=D, B=B, P=P, n_tokens=tuple(n), deltas=tuple(deltas),
                          rho0s=tuple(rho0s), tag_set=tag_set, mix=[1.0] * len(tag_set),
                          repair_frac=float(r.choice([0.0, 0.1, 0.3])), out_dtype=out, theta=theta,
                          outlier_pairs=int(r.integers(0, 2)))
    style = int(r.integers(0, 2))
    R = int(16 * r.integers(1, D // 16 + 1))
    scaled = bool(r.random() < 0.3)
    layout = int(r.integers(0, 2))
    case.shape = dataclasses.replace(case.shape, rope_style=style, rotary_dim=0 if R == D else R,
                                     inv_freq=wl.llama3_inv_freq(theta, R) if scaled else None, kv_layout=layout)
    return case


def describe(case) -> str:
    s = case.shape
    return (f"L{s.num_layers} H{s.num_kv_heads} D{s.head_dim} B{s.block_tokens} P{s.page_size} "
            f"out={'bf16' if s.out_dtype else 'fp16'} rope={'interleaved' if s.rope_style else 'half'} "
            f"R={s.rotary_dim or s.head_dim} scaled={s.inv_freq is not None} theta={s.rope_theta:g} "
            f"kv={'paired' if s.kv_layout else 'separate'} "
            f"reqs={[(q.suffix_tokens, q.delta, q.dst_row0) for q in case.requests]} "
            f"tags={sorted(set(int(t) for q in case.requests for t in q.tags))}")


# Configurations at the limits the planner accepts: rows of H * D = 4096
# elements (the largest), head_dim 512 (the largest), blocks of 1024 tokens
# (the largest), one-token and 1024-token pages.
LIMIT_CASES = {
    "hd4096_h32_d128": dict(L=1, H=32, D=128, B=8, P=8, n_tokens=(61, 17), deltas=(-300, 7), rho0s=(5, 3)),
    "hd4096_h8_d512": dict(L=2, H=8, D=512, B=4, P=2, n_tokens=(23,), deltas=(9000,), rho0s=(1,)),
    "b1024_p1024": dict(L=1, H=2, D=64, B=1024, P=1024, n_tokens=(2500,), deltas=(-5,), rho0s=(1000,)),
    "b1024_p1": dict(L=1, H=1, D=32, B=1024, P=1, n_tokens=(1100,), deltas=(3,), rho0s=(2,)),
}


def limit_case(name: str) -> "wl.Case":
    case = wl.make_custom(77, tag_set=(0, 1, 2, 3), mix=(1, 1, 1, 1), repair_frac=0.2, out_dtype=wl.OUT_BF16,
                          outlier_pairs=1, **LIMIT_CASES[name])
    if name.startswith("b1024"):  # the largest blocks on paired pages too
        case.shape = dataclasses.replace(case.shape, kv_layout=wl.KV_PAIRED)
    return case
