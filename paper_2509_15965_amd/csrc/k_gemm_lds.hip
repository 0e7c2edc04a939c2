// k_gemm_lds.hip -- Y = X . W^T for batches of more than 64 rows (decode at
// large batch, prefill): LDS-tiled MFMA GEMM.
//
// Workgroup tile BM x BN (weight rows) x 64 (k), 4 waves in a 2 x 2 grid, each
// wave (BM/2) x (BN/2) of 16x16x32 bf16 MFMA tiles.  Global tiles go through
// registers into a double-buffered, row-padded LDS (72 elements per 64-wide
// row, so the 16-byte fragment reads of 16 rows hit distinct banks); the next
// k tile's global loads are in flight while the current one feeds the MFMAs,
// with one barrier per k tile.
//
// Tile order is XCD-aware: workgroup w runs on XCD w % 8, and each XCD walks
// its own weight tiles (n % 8 == xcd) with groups of up to 8 M tiles
// back-to-back, so the M tiles that share a weight tile run together and
// read it from that XCD's L2 instead of HBM.
#include "rl_device.h"
#include "rl_internal.h"

namespace rl {

namespace {

template <int BM, int BN, int EPI, bool SPLIT>
__global__ void __launch_bounds__(256) gemm_lds_kernel(GemmArgs p, int ksplit, int m_tiles, int n_tiles,
                                                       int gm) {
    constexpr int BK = 64, LDK = BK + 8;
    constexpr int TM = BM / 2, TN = BN / 2;
    constexpr int MT = TM / 16, NT = TN / 16;
    constexpr int AL = BM / 32, BL = BN / 32;   // 16-byte global loads per thread
    __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * LDK];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN * LDK];

    const int w = blockIdx.x;
    const int xcd = w & 7, j = w >> 3;
    const int ntx = (n_tiles + 7) >> 3;
    const int grp = j / (gm * ntx);
    const int rem = j - grp * gm * ntx;
    const int m_tile = grp * gm + rem % gm;
    const int n_tile = (rem / gm) * 8 + xcd;
    if (m_tile >= m_tiles || n_tile >= n_tiles) return;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int r16 = lane & 15, kq = lane >> 4;
    const int M = p.M, Nw = p.Nw, K = p.K;
    const int m0 = m_tile * BM;

    // weight row held by LDS B row b (SwiGLU: each wave's tiles pair gate and up rows)
    auto wrow = [&](int b, bool* ok) -> int {
        if (EPI == EPI_SWIGLU) {
            const int wv = b / TN, u = b - wv * TN;
            const int c0 = n_tile * (BN / 2) + wv * (TN / 2);
            const int c = u < TN / 2 ? c0 + u : c0 + u - TN / 2;
            *ok = c < p.F;
            return u < TN / 2 ? c : p.F + c;
        } else {
            const int n = n_tile * BN + b;
            *ok = n < Nw;
            return n;
        }
    };

    const int kb = blockIdx.y * ksplit;
    const int ke = min(K, kb + ksplit);
    const int nk = (ke - kb + BK - 1) / BK;

    const uint16_t* A = static_cast<const uint16_t*>(p.A);
    const uint16_t* W = static_cast<const uint16_t*>(p.W);
    const int lr = tid >> 3, lk = (tid & 7) * 8;
    const uint16_t* ag[AL];
    bool aok[AL];
#pragma unroll
    for (int i = 0; i < AL; ++i) {
        const int m = m0 + lr + 32 * i;
        aok[i] = m < M;
        ag[i] = A + static_cast<size_t>(aok[i] ? m : 0) * p.lda + lk;
    }
    const uint16_t* bg[BL];
    bool bok[BL];
#pragma unroll
    for (int i = 0; i < BL; ++i) {
        bool ok;
        const int n = wrow(lr + 32 * i, &ok);
        bok[i] = ok;
        bg[i] = W + static_cast<size_t>(ok ? n : 0) * p.ldw + lk;
    }

    const u32x4 zero = {0u, 0u, 0u, 0u};
    u32x4 ra[AL], rb[BL];
    auto gload = [&](int k0) {
        const bool kok = k0 + lk < ke;
#pragma unroll
        for (int i = 0; i < AL; ++i) ra[i] = (aok[i] && kok) ? ld16(ag[i] + k0) : zero;
#pragma unroll
        for (int i = 0; i < BL; ++i) rb[i] = (bok[i] && kok) ? ld16(bg[i] + k0) : zero;
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < AL; ++i)
            *reinterpret_cast<u32x4*>(&As[buf][(lr + 32 * i) * LDK + lk]) = ra[i];
#pragma unroll
        for (int i = 0; i < BL; ++i)
            *reinterpret_cast<u32x4*>(&Bs[buf][(lr + 32 * i) * LDK + lk]) = rb[i];
    };

    f32x4 acc[MT][NT];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[i][t] = f32x4{0.f, 0.f, 0.f, 0.f};

    if (nk > 0) {
        gload(kb);
        sstore(0);
    }
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt & 1;
        const bool more = kt + 1 < nk;
        if (more) gload(kb + (kt + 1) * BK);
        const uint16_t* as = &As[cur][(wm * TM + r16) * LDK + 8 * kq];
        const uint16_t* bs = &Bs[cur][(wn * TN + r16) * LDK + 8 * kq];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            u32x4 af[MT], bf[NT];
#pragma unroll
            for (int i = 0; i < MT; ++i) af[i] = *reinterpret_cast<const u32x4*>(as + 16 * i * LDK + 32 * ks);
#pragma unroll
            for (int t = 0; t < NT; ++t) bf[t] = *reinterpret_cast<const u32x4*>(bs + 16 * t * LDK + 32 * ks);
#pragma unroll
            for (int i = 0; i < MT; ++i)
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    acc[i][t] = mfma16x16x32(as_bf16x8(af[i]), as_bf16x8(bf[t]), acc[i][t]);
        }
        if (more) sstore(cur ^ 1);
        __syncthreads();
    }

    // epilogue: acc[i][t][e] is row m0 + wm*TM + 16i + 4kq + e, LDS B row wn*TN + 16t + r16
    int nrow[NT];
    bool nok[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) nrow[t] = wrow(wn * TN + 16 * t + r16, &nok[t]);
#pragma unroll
    for (int i = 0; i < MT; ++i) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int m = m0 + wm * TM + 16 * i + 4 * kq + e;
            if (m >= M) continue;
            if (SPLIT) {
                float* dst = p.partial + (static_cast<size_t>(blockIdx.y) * M + m) * Nw;
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    if (nok[t]) dst[nrow[t]] = acc[i][t][e];
            } else if (EPI == EPI_F32) {
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    if (nok[t]) p.out_f32[static_cast<size_t>(m) * p.ldo + nrow[t]] = acc[i][t][e];
            } else if (EPI == EPI_RESID) {
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    if (nok[t]) p.resid[static_cast<size_t>(m) * p.ldr + nrow[t]] += acc[i][t][e];
            } else {
                uint16_t* act = static_cast<uint16_t*>(p.act);
#pragma unroll
                for (int t = 0; t < NT / 2; ++t) {
                    if (!nok[t]) continue;
                    const float g = acc[i][t][e], u = acc[i][t + NT / 2][e];
                    const float silu = g / (1.0f + expf(-g));
                    act[static_cast<size_t>(m) * p.ld_act + nrow[t]] = f32_to_bf16(silu * u);
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Direct-to-LDS ring variant (K a multiple of 32).  global_load_lds_dwordx4
// moves each 16-byte chunk from global memory straight into LDS, so no
// staging registers are needed and a ring of S k-stages (32 wide) keeps
// S - 2 stages of HBM traffic in flight while the MFMAs consume another; the
// ring fills most of the 160 KB LDS.  LDS rows are 32 elements (64 bytes);
// the four 16-byte chunks of row r sit at chunk ^ ((r / 2) % 4), so one DMA
// instruction fills 16 whole rows (1 KB, lane i -> bytes 16i) and the
// fragment reads of 8 consecutive rows hit 8 distinct bank groups.  Each
// stage is guarded by one barrier; the next stage's fragments are read under
// the current stage's MFMAs.  Rows past M or past the weight are loaded from a
// clamped valid row and their outputs are never stored.
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void lds_void_t;

__device__ __forceinline__ void dma16(const uint16_t* g, uint8_t* lds_wave_base) {
    __builtin_amdgcn_global_load_lds(static_cast<const void*>(g), (lds_void_t*)(lds_wave_base), 16, 0, 0);
}

// s_waitcnt vmcnt(n) with the other counters left alone (gfx9 encoding)
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// wait until at most `outstanding` (0..4) later stages of Q DMA ops each are pending
template <int Q>
__device__ __forceinline__ void wait_stages(int outstanding) {
    switch (outstanding) {
        case 0: wait_vm<0>(); break;
        case 1: wait_vm<Q>(); break;
        case 2: wait_vm<2 * Q>(); break;
        case 3: wait_vm<3 * Q>(); break;
        default: wait_vm<4 * Q>(); break;
    }
}

template <int BM, int BN, int WM, int S, int EPI, bool SPLIT>
__global__ void __launch_bounds__(256) gemm_dma_kernel(GemmArgs p, int ksplit, int m_tiles, int n_tiles,
                                                       int gm) {
    constexpr int BK = 32, ROWB = 64;
    constexpr int WN = 4 / WM;
    constexpr int TM = BM / WM, TN = BN / WN;
    constexpr int MT = TM / 16, NT = TN / 16;
    constexpr int STAGE = (BM + BN) * ROWB;
    constexpr int AQ = BM / 64, BQ = BN / 64;   // DMA instructions (16 rows each) per wave per stage
    constexpr int Q = AQ + BQ;
    static_assert(BM % 64 == 0 && BN % 64 == 0, "tile rows must fill whole DMA instructions");
    static_assert(S >= 3 && S - 2 <= 4 && Q * 4 < 64, "vmcnt range");
    __shared__ __attribute__((aligned(1024))) uint8_t smem[S * STAGE];

    const int w = blockIdx.x;
    const int xcd = w & 7, j = w >> 3;
    const int ntx = (n_tiles + 7) >> 3;
    const int grp = j / (gm * ntx);
    const int rem = j - grp * gm * ntx;
    const int m_tile = grp * gm + rem % gm;
    const int n_tile = (rem / gm) * 8 + xcd;
    if (m_tile >= m_tiles || n_tile >= n_tiles) return;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    const int r16 = lane & 15, kq = lane >> 4;
    const int M = p.M, Nw = p.Nw, K = p.K;
    const int m0 = m_tile * BM;

    auto wrow = [&](int b, bool* ok) -> int {
        if (EPI == EPI_SWIGLU) {
            const int wv = b / TN, u = b - wv * TN;
            const int c0 = n_tile * (BN / 2) + wv * (TN / 2);
            const int c = u < TN / 2 ? c0 + u : c0 + u - TN / 2;
            *ok = c < p.F;
            return u < TN / 2 ? c : p.F + c;
        } else {
            const int n = n_tile * BN + b;
            *ok = n < Nw;
            return n;
        }
    };

    const int kb = blockIdx.y * ksplit;
    const int ke = min(K, kb + ksplit);
    const int nk = (ke - kb) / BK;

    const uint16_t* A = static_cast<const uint16_t*>(p.A);
    const uint16_t* W = static_cast<const uint16_t*>(p.W);
    // this lane's DMA source: row 16g + lane/4, original chunk (lane%4) ^ ((lane/8)%4)
    const int lrow = lane >> 2, lch = (lane & 3) ^ ((lane >> 3) & 3);
    uint32_t aoff[AQ], boff[BQ];
#pragma unroll
    for (int q = 0; q < AQ; ++q) {
        int m = m0 + 16 * (wave * AQ + q) + lrow;
        m = m < M ? m : M - 1;
        aoff[q] = static_cast<uint32_t>(m) * static_cast<uint32_t>(p.lda) + 8u * lch;
    }
#pragma unroll
    for (int q = 0; q < BQ; ++q) {
        bool ok;
        int n = wrow(16 * (wave * BQ + q) + lrow, &ok);
        n = ok ? n : 0;
        boff[q] = static_cast<uint32_t>(n) * static_cast<uint32_t>(p.ldw) + 8u * lch;
    }
    auto issue = [&](int stage, int k0) {
        uint8_t* abase = smem + (stage % S) * STAGE;
        uint8_t* bbase = abase + BM * ROWB;
#pragma unroll
        for (int q = 0; q < AQ; ++q) dma16(A + aoff[q] + k0, abase + (wave * AQ + q) * 1024);
#pragma unroll
        for (int q = 0; q < BQ; ++q) dma16(W + boff[q] + k0, bbase + (wave * BQ + q) * 1024);
    };

    f32x4 acc[MT][NT];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[i][t] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int sw = (kq ^ ((r16 >> 1) & 3)) * 16;
    const int arow = (wm * TM + r16) * ROWB + sw;
    const int brow = BM * ROWB + (wn * TN + r16) * ROWB + sw;
    auto frag_a = [&](int stage, int i) {
        return *reinterpret_cast<const u32x4*>(smem + (stage % S) * STAGE + arow + 16 * i * ROWB);
    };
    auto frag_b = [&](int stage, int t) {
        return *reinterpret_cast<const u32x4*>(smem + (stage % S) * STAGE + brow + 16 * t * ROWB);
    };

    // prologue: stages 0 .. S-2 in flight, then stage 0 resident
#pragma unroll
    for (int st = 0; st < S - 1; ++st)
        if (st < nk) issue(st, kb + st * BK);
    wait_stages<Q>(min(S - 2, nk - 1));
    __syncthreads();
    u32x4 fa[MT], fb[NT];
#pragma unroll
    for (int i = 0; i < MT; ++i) fa[i] = frag_a(0, i);
#pragma unroll
    for (int t = 0; t < NT; ++t) fb[t] = frag_b(0, t);

    for (int kt = 0; kt < nk; ++kt) {
        const bool has_next = kt + 1 < nk;
        if (has_next) {
            wait_stages<Q>(min(S - 3, nk - 2 - kt));   // stage kt+1 resident
            __syncthreads();                               // and every wave is done with stage kt-1
            if (kt + S - 1 < nk) issue(kt + S - 1, kb + (kt + S - 1) * BK);
        }
        const int nxt = has_next ? kt + 1 : kt;
        u32x4 ga[MT], gb[NT];
#pragma unroll
        for (int i = 0; i < MT; ++i) ga[i] = frag_a(nxt, i);
#pragma unroll
        for (int t = 0; t < NT; ++t) gb[t] = frag_b(nxt, t);
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int t = 0; t < NT; ++t)
                acc[i][t] = mfma16x16x32(as_bf16x8(fa[i]), as_bf16x8(fb[t]), acc[i][t]);
        constexpr int NRD = MT + NT;
        constexpr int R = (MT * NT) / NRD > 0 ? (MT * NT) / NRD : 1;
#pragma unroll
        for (int g = 0; g < NRD; ++g) {
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, R, 0);
        }
#pragma unroll
        for (int i = 0; i < MT; ++i) fa[i] = ga[i];
#pragma unroll
        for (int t = 0; t < NT; ++t) fb[t] = gb[t];
    }

    int nrow[NT];
    bool nok[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) nrow[t] = wrow(wn * TN + 16 * t + r16, &nok[t]);
#pragma unroll
    for (int i = 0; i < MT; ++i) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int m = m0 + wm * TM + 16 * i + 4 * kq + e;
            if (m >= M) continue;
            if (SPLIT) {
                float* dst = p.partial + (static_cast<size_t>(blockIdx.y) * M + m) * Nw;
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    if (nok[t]) dst[nrow[t]] = acc[i][t][e];
            } else if (EPI == EPI_F32) {
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    if (nok[t]) p.out_f32[static_cast<size_t>(m) * p.ldo + nrow[t]] = acc[i][t][e];
            } else if (EPI == EPI_RESID) {
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    if (nok[t]) p.resid[static_cast<size_t>(m) * p.ldr + nrow[t]] += acc[i][t][e];
            } else {
                uint16_t* act = static_cast<uint16_t*>(p.act);
#pragma unroll
                for (int t = 0; t < NT / 2; ++t) {
                    if (!nok[t]) continue;
                    const float g = acc[i][t][e], u = acc[i][t + NT / 2][e];
                    const float silu = g / (1.0f + expf(-g));
                    act[static_cast<size_t>(m) * p.ld_act + nrow[t]] = f32_to_bf16(silu * u);
                }
            }
        }
    }
}

template <int BM, int BN, int WM, int S>
hipError_t launch_dma(const GemmArgs& a, const GemmPlan& p, hipStream_t s) {
    const int m_tiles = (a.M + BM - 1) / BM;
    const int n_out = a.epi == EPI_SWIGLU ? a.F : a.Nw;
    const int bno = a.epi == EPI_SWIGLU ? BN / 2 : BN;
    const int n_tiles = (n_out + bno - 1) / bno;
    const int gm = m_tiles < 8 ? m_tiles : 8;
    const int ntx = (n_tiles + 7) / 8;
    const int groups = (m_tiles + gm - 1) / gm;
    dim3 grid(8 * ntx * groups * gm, p.splits), block(256);
    if (p.splits > 1) {
        if (a.epi == EPI_SWIGLU)
            hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, WM, S, EPI_SWIGLU, true>), grid, block, 0, s, a, p.ksplit, m_tiles, n_tiles, gm);
        else
            hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, WM, S, EPI_F32, true>), grid, block, 0, s, a, p.ksplit, m_tiles, n_tiles, gm);
    } else if (a.epi == EPI_F32) {
        hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, WM, S, EPI_F32, false>), grid, block, 0, s, a, p.ksplit, m_tiles, n_tiles, gm);
    } else if (a.epi == EPI_RESID) {
        hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, WM, S, EPI_RESID, false>), grid, block, 0, s, a, p.ksplit, m_tiles, n_tiles, gm);
    } else {
        hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, WM, S, EPI_SWIGLU, false>), grid, block, 0, s, a, p.ksplit, m_tiles, n_tiles, gm);
    }
    return hipGetLastError();
}

template <int BM, int BN>
hipError_t launch_tile(const GemmArgs& a, const GemmPlan& p, hipStream_t s) {
    const int m_tiles = (a.M + BM - 1) / BM;
    const int n_out = a.epi == EPI_SWIGLU ? a.F : a.Nw;
    const int bno = a.epi == EPI_SWIGLU ? BN / 2 : BN;
    const int n_tiles = (n_out + bno - 1) / bno;
    const int gm = m_tiles < 8 ? m_tiles : 8;
    const int ntx = (n_tiles + 7) / 8;
    const int groups = (m_tiles + gm - 1) / gm;
    dim3 grid(8 * ntx * groups * gm, p.splits), block(256);
    if (p.splits > 1) {
        if (a.epi == EPI_SWIGLU)
            hipLaunchKernelGGL((gemm_lds_kernel<BM, BN, EPI_SWIGLU, true>), grid, block, 0, s, a, p.ksplit, m_tiles, n_tiles, gm);
        else
            hipLaunchKernelGGL((gemm_lds_kernel<BM, BN, EPI_F32, true>), grid, block, 0, s, a, p.ksplit, m_tiles, n_tiles, gm);
    } else if (a.epi == EPI_F32) {
        hipLaunchKernelGGL((gemm_lds_kernel<BM, BN, EPI_F32, false>), grid, block, 0, s, a, p.ksplit, m_tiles, n_tiles, gm);
    } else if (a.epi == EPI_RESID) {
        hipLaunchKernelGGL((gemm_lds_kernel<BM, BN, EPI_RESID, false>), grid, block, 0, s, a, p.ksplit, m_tiles, n_tiles, gm);
    } else {
        hipLaunchKernelGGL((gemm_lds_kernel<BM, BN, EPI_SWIGLU, false>), grid, block, 0, s, a, p.ksplit, m_tiles, n_tiles, gm);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_bf16_lds(const GemmArgs& a, const GemmPlan& p, hipStream_t s) {
    if (a.M <= 0) return hipSuccess;
    if (p.variant == kLdsVariant256x256) return launch_dma<256, 256, 2, 5>(a, p, s);
    if (p.variant == kDmaVariant128) return launch_dma<128, 256, 2, 6>(a, p, s);
    if (p.variant == kLdsVariant256) return launch_tile<256, 128>(a, p, s);
    return launch_tile<128, 128>(a, p, s);
}

}  // namespace rl
