"""One decode step over a compacted cache (stepkv_decode_attention) against textbook
attention (the oracle's decode_attention), within 2e-3 of each row's largest magnitude.

The caches here are seeded random rows laid out as the compaction writes them, with
ragged retained counts (0, 1, and several 256-row splits) and query groups of 1, 4, 7
12, 16 and 32 heads per KV head (the last wider than the grouped kernel's 16, so the
per-head kernel), one case whose logits spread over ~100 nats, so the running
reference of each head moves in the middle of a split, one whose sequences are far
longer than what they retain (the split count then comes from out_rows, and here every
split that bound allows holds rows), one whose out_rows cuts the last sequences
short (rows at or past out_rows are not read), and one large enough for splits of 1024
rows instead of 512."""
import math
import zlib

import numpy as np
import pytest

import oracle as O
from paper_2609_22158_amd import binding as B
from synth import f32_to_bf16_bits
from tests.gpu_cases import log

pytestmark = pytest.mark.gpu

CASES = {
    # name: (L, Hq, Hkv, d, retained rows per sequence, out_rows slack, key scale[,
    #        most tokens a sequence had beyond its retained rows])
    "g4_d128_splits": (2, 32, 8, 128, [1536, 700, 1, 0, 257], 0, 3.0),
    "g7_d128": (2, 28, 4, 128, [2560, 31, 513], 5, 3.0),
    "g1_d64": (3, 4, 4, 64, [300, 64, 0, 1000], 0, 3.0),
    "g16_d128": (1, 32, 2, 128, [900, 3], 0, 3.0),
    "g2_d64": (1, 4, 2, 64, [256, 255, 257], 0, 3.0),
    "g8_d64": (2, 16, 2, 64, [1100, 17, 16, 15], 0, 3.0),
    "g12_d128": (1, 24, 2, 128, [530, 47], 0, 3.0),  # 12 of the 16 MFMA columns in use
    "g32_d128_wide": (1, 32, 1, 128, [700, 2], 0, 3.0),  # wider than 16: the per-head kernel
    # logits spread over ~100 nats, so the per-head reference moves within a split
    "g7_d128_peaky": (1, 14, 2, 128, [1400, 600], 0, 40.0),
    # 4 x 2 splits of 512 rows = floor(out_rows / 512) + S: the bound is met exactly
    "g8_d128_tight": (1, 16, 2, 128, [513, 513, 513, 513], 0, 3.0, 20000),
    # out_rows = 950: the second sequence keeps 250 rows, the third none
    "g4_d128_short": (1, 8, 2, 128, [700, 600, 300], -650, 3.0),
    # L * Hkv * floor(out_rows / 1024) = 1632 >= 2 * 768: splits of 1024 rows
    "g2_d64_long": (2, 16, 8, 64, [30000, 25000, 1, 50000], 0, 3.0),
}


@pytest.mark.parametrize("cid", list(CASES))
def test_decode_matches_textbook_attention(cid):
    import torch

    L, Hq, Hkv, d, rows, slack, kscale, *extra = CASES[cid]
    extra = extra[0] if extra else 50
    G = Hq // Hkv
    S = len(rows)
    rng = np.random.default_rng(zlib.crc32(cid.encode()))
    cu_ret = np.concatenate([[0], np.cumsum(rows)]).astype(np.int32)
    out_rows = int(cu_ret[-1]) + slack
    seqlens = [r + int(rng.integers(0, extra)) for r in rows]  # the cache each came from was longer
    cu_seq = np.concatenate([[0], np.cumsum(seqlens)]).astype(np.int32)
    pb = B.Problem(L, Hq, Hkv, d, 1, cu_seq, np.zeros(S + 1, np.int32))
    qb = f32_to_bf16_bits(rng.standard_normal((L, S, Hq, d)).astype(np.float32))
    kb = f32_to_bf16_bits((rng.standard_normal((L, Hkv, out_rows, d)) / math.sqrt(d) * kscale).astype(np.float32))
    vb = f32_to_bf16_bits(rng.standard_normal((L, Hkv, out_rows, d)).astype(np.float32))
    log(f"[decode {cid}] L={L} Hq={Hq} Hkv={Hkv} d={d} rows={rows}")
    out = B.decode_attention(pb, B.bf16_from_bits(qb), B.bf16_from_bits(kb), B.bf16_from_bits(vb),
                             torch.from_numpy(cu_ret).cuda(), out_rows).cpu().numpy()
    scale = 1.0 / math.sqrt(d)
    for l in range(L):
        for s in range(S):
            a, b = min(int(cu_ret[s]), out_rows), min(int(cu_ret[s + 1]), out_rows)
            for hq in range(Hq):
                got = out[l, s, hq]
                if b == a:
                    assert np.all(got == 0), (l, s, hq)
                    continue
                h = hq // G
                ref = O.decode_attention(O.decode_bf16(qb[l, s, hq]), O.decode_bf16(kb[l, h, a:b]),
                                         O.decode_bf16(vb[l, h, a:b]), scale)
                tol = 2e-3 * max(float(np.abs(ref).max()), 1e-30)
                assert np.abs(got - ref).max() <= tol, (cid, l, s, hq, np.abs(got - ref).max(), tol)
