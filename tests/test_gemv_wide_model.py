"""CPU model of the wide GEMV's index math (gemv_wide_kernel and
launch_gemv_wide in paper_2509_15965_amd/csrc/k_gemm.hip).

A workgroup owns four 16-row weight groups (SwiGLU: 8 gate rows and the
matching 8 up rows each) and one K slice; wave w takes the w-th quarter of the
slice, lane (r16, kq) loads 8 k values at kk + 8 kq for kk stepping by 32 while
kk + 8 kq < the wave's end.  This model replays those formulas for every
workgroup, wave and lane and checks, for the shapes the decoder uses and the
split counts a plan can ask for:
  - every weight row read exists (row < Nw) and every k read lies in [0, K);
  - each weight element (n, k) is multiplied exactly once over the whole grid;
  - every activation row read is < M, and M fits the MR tiles of 16 rows;
  - every output store is in bounds: the split-K partials within
    splits x M x Nw, SwiGLU outputs within F, and each output (m, n) is
    written exactly once per split.
A mapping with the up-row offset dropped must fail it.
"""
import numpy as np
import pytest


def cdiv(a, b):
    return (a + b - 1) // b


def plan(K, s):
    ks = cdiv(cdiv(K, s), 64) * 64 if s > 1 else K
    return ks, cdiv(K, ks)


def rows_of(g, t, r16, epi, F, Nw, up_offset=True):
    """Weight rows and validity of lanes r16 in weight group t of workgroups g
    (arrays broadcast: g down, r16 across)."""
    if epi == "swiglu":
        c = (g * 4 + t) * 8 + (r16 & 7)
        ok = c < F
        n = np.where(r16 < 8, c, (F if up_offset else 0) + c)
    else:
        n = (g * 4 + t) * 16 + r16
        ok = n < Nw
    return n, ok


def replay(M, Nw, K, epi, F, s, up_offset=True):
    ks, splits = plan(K, s)
    groups = cdiv(F, 32) if epi == "swiglu" else cdiv(Nw, 64)
    kw = cdiv(cdiv(ks, 4), 64) * 64
    MR = 1 if M <= 16 else 2 if M <= 32 else 4
    assert MR * 16 >= M
    lane = np.arange(64)
    r16, kq = lane & 15, lane >> 4
    g = np.arange(groups)[:, None]
    reads, writes = [], []   # flat indices: 8-element weight fragments, outputs (split, m, n)
    for t in range(4):
        n, ok = rows_of(g, t, r16[None, :], epi, F, Nw, up_offset)
        assert np.all((n[ok] >= 0) & (n[ok] < Nw))
        for y in range(splits):
            ks0 = y * ks
            ks1 = min(K, ks0 + ks)
            for w in range(4):
                kb = ks0 + w * kw
                ke = min(ks1, kb + kw)
                for kk in range(kb, ke, 32):
                    k = np.broadcast_to(kk + 8 * kq[None, :], n.shape)
                    sel = ok & (k < ke)
                    assert np.all(k[sel] + 8 <= K)
                    reads.append(n[sel] * (K // 8) + k[sel] // 8)
            # stores: lane holds rows 16 i + 4 kq + e of column n
            for i in range(MR):
                for e in range(4):
                    m = np.broadcast_to(16 * i + 4 * kq[None, :] + e, n.shape)
                    sel = ok & (m < M)
                    if epi == "swiglu" and splits == 1:
                        sel &= r16[None, :] < 8          # the gate lane writes the SwiGLU output
                        assert np.all(n[sel] < F)
                    writes.append((y * M + m[sel]) * Nw + n[sel])
    reads = np.bincount(np.concatenate(reads), minlength=Nw * K // 8).reshape(Nw, K // 8)
    writes = np.bincount(np.concatenate(writes), minlength=splits * M * Nw).reshape(splits, M, Nw)
    return reads, writes, splits


SHAPES = [  # (Nw, K, epilogue, F): the test decoder, then the 7B widths
    (1536, 512, "f32", 0), (512, 1024, "resid", 0), (2048, 512, "swiglu", 1024), (1032, 512, "f32", 0),
    (4608, 3584, "f32", 0), (3584, 3584, "resid", 0), (37888, 3584, "swiglu", 18944),
]


@pytest.mark.parametrize("Nw,K,epi,F", SHAPES)
@pytest.mark.parametrize("M", [1, 5, 16, 17, 40, 64])
def test_wide_gemv_covers_every_product_once(Nw, K, epi, F, M):
    for s in (1, 2, 3, 8):
        reads, writes, splits = replay(M, Nw, K, epi, F, s)
        assert np.all(reads == 1), (s, np.unique(reads))
        if epi == "swiglu" and splits == 1:
            assert np.all(writes[0, :, :F] == 1) and not writes[0, :, F:].any()
        else:
            assert np.all(writes == 1), s


def test_wide_gemv_model_catches_a_missing_up_offset():
    reads, _, _ = replay(8, 2048, 512, "swiglu", 1024, 1, up_offset=False)
    assert not np.all(reads == 1)
