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

#include <algorithm>
#include <type_traits>

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
                    act[static_cast<size_t>(m) * p.ld_act + nrow[t]] = f32_to_bf16(swiglu_bf16(g, u));
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Direct-to-LDS ring variant (K a multiple of 32).  global_load_lds_dwordx4
// moves each 16-byte chunk from global memory straight into LDS, so no
// staging registers are needed and a ring of S k-stages (32 wide) keeps
// S - 2 to S - 1 stages of HBM traffic in flight while the MFMAs consume
// another; the ring fills the 160 KB LDS.  LDS rows are 32 elements (64 bytes);
// the four 16-byte chunks of row r sit at chunk ^ ((r / 4) % 4), so one DMA
// instruction fills 16 whole rows (1 KB, lane i -> bytes 16i) and the 32x32
// fragment reads (32 rows x 2 chunks per instruction) are free of bank
// conflicts.  Each stage is guarded by one barrier; the next stage's
// fragments are read under the current stage's MFMAs, into the other half of
// a statically alternating register pair (the k loop is unrolled by two).
// Rows past M or past the weight are loaded from a clamped valid row and
// their outputs are never stored.
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void lds_void_t;

__device__ __forceinline__ void dma16(const uint16_t* g, uint8_t* lds_wave_base) {
    __builtin_amdgcn_global_load_lds(static_cast<const void*>(g), (lds_void_t*)(lds_wave_base), 16, 0, 0);
}

// Same, from a wave-uniform base plus a 32-bit per-lane byte offset: the
// address then stays in the scalar-base form of the instruction (no 64-bit
// per-lane address arithmetic per issue).
__device__ __forceinline__ void dma16_off(const uint8_t* base, uint32_t off, uint8_t* lds_wave_base) {
    __builtin_amdgcn_global_load_lds(static_cast<const void*>(base + off), (lds_void_t*)(lds_wave_base), 16, 0, 0);
}

// s_waitcnt vmcnt(n) with the other counters left alone (gfx9 encoding)
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// wait until at most `outstanding` (0..MAXS) later stages of Q DMA ops each are pending
template <int Q, int MAXS>
__device__ __forceinline__ void wait_stages(int outstanding) {
    static_assert(MAXS <= 5 && Q * MAXS < 64, "vmcnt range");
    switch (outstanding) {
        case 0: wait_vm<0>(); break;
        case 1: wait_vm<Q>(); break;
        case 2: wait_vm<(2 <= MAXS ? 2 : MAXS) * Q>(); break;
        case 3: wait_vm<(3 <= MAXS ? 3 : MAXS) * Q>(); break;
        case 4: wait_vm<(4 <= MAXS ? 4 : MAXS) * Q>(); break;
        default: wait_vm<MAXS * Q>(); break;
    }
}

template <int BM, int BN, int WM, int NW, int S, int EPI, bool SPLIT>
__global__ void __launch_bounds__(64 * NW) gemm_dma_kernel(GemmArgs p, int ksplit, int m_tiles, int n_tiles, int n0,
                                                           int gm) {
    constexpr int BK = 32, ROWB = 64;
    constexpr int WN = NW / WM;
    constexpr int TM = BM / WM, TN = BN / WN;
    constexpr int MT = TM / 32, NT = TN / 32;
    constexpr int STAGE = (BM + BN) * ROWB;
    constexpr int AQ = BM / (16 * NW), BQ = BN / (16 * NW);   // DMA instructions (16 rows each) per wave per stage
    constexpr int Q = AQ + BQ;
    static_assert(BM % (16 * NW) == 0 && BN % (16 * NW) == 0, "tile rows must fill whole DMA instructions");
    static_assert(TM % 32 == 0 && TN % 64 == 0, "wave tile must hold whole 32x32 tiles (and gate/up pairs)");
    static_assert(S >= 3 && S - 1 <= 5, "ring depth");
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
    const int r32 = lane & 31, kh = lane >> 5;
    const int M = p.M, Nw = p.Nw, K = p.K;
    const int m0 = m_tile * BM;

    auto wrow = [&](int b, bool* ok) -> int {
        if (EPI == EPI_SWIGLU) {
            const int wv = b / TN, u = b - wv * TN;
            const int c0 = n0 + n_tile * (BN / 2) + wv * (TN / 2);
            const int c = u < TN / 2 ? c0 + u : c0 + u - TN / 2;
            *ok = c < p.F;
            return u < TN / 2 ? c : p.F + c;
        } else {
            const int n = n0 + n_tile * BN + b;
            *ok = n < Nw;
            return n;
        }
    };

    const int kb = blockIdx.y * ksplit;
    const int ke = min(K, kb + ksplit);
    const int nk = (ke - kb) / BK;

    const uint16_t* A = static_cast<const uint16_t*>(p.A);
    const uint16_t* W = static_cast<const uint16_t*>(p.W);
    // this lane's DMA source: row 16g + lane/4, original chunk (lane%4) ^ ((row/4)%4)
    const int lrow = lane >> 2, lch = (lane & 3) ^ ((lane >> 4) & 3);
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

    f32x16 acc[MT][NT];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][t][e] = 0.f;

    // lane (r32, kh) reads k chunk 2 ks + kh (16 bytes) of its row in sub-step ks;
    // every fragment row is r32 plus a multiple of 32, so the swizzle depends on r32 only
    const int sw0 = ((0 + kh) ^ ((r32 >> 2) & 3)) * 16;
    const int sw1 = ((2 + kh) ^ ((r32 >> 2) & 3)) * 16;
    // per-lane byte offsets inside a stage; tile i / t adds an immediate 32 rows
    const uint32_t la0 = (wm * TM + r32) * ROWB + sw0, la1 = (wm * TM + r32) * ROWB + sw1;
    const uint32_t lb0 = (BM + wn * TN + r32) * ROWB + sw0, lb1 = (BM + wn * TN + r32) * ROWB + sw1;
    auto frag = [&](uint32_t lane_stage, int imm) {
        return *reinterpret_cast<const u32x4*>(smem + lane_stage + imm);
    };
    // fragments of one k sub-step (16 wide) of a stage
    auto load_half = [&](int stage, int ks, u32x4 (&fa)[MT], u32x4 (&fb)[NT]) {
        const uint32_t so = static_cast<uint32_t>(stage % S) * STAGE;
        const uint32_t a = so + (ks ? la1 : la0), b = so + (ks ? lb1 : lb0);
#pragma unroll
        for (int i = 0; i < MT; ++i) fa[i] = frag(a, 32 * i * ROWB);
#pragma unroll
        for (int t = 0; t < NT; ++t) fb[t] = frag(b, 32 * t * ROWB);
    };
    auto mma_half = [&](const u32x4 (&fa)[MT], const u32x4 (&fb)[NT]) {
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int t = 0; t < NT; ++t)
                acc[i][t] = mfma32x32x16(as_bf16x8(fa[i]), as_bf16x8(fb[t]), acc[i][t]);
        constexpr int NRD = MT + NT, NMF = MT * NT;
        constexpr int R = NMF / NRD > 0 ? NMF / NRD : 1;
#pragma unroll
        for (int g = 0; g < NRD; ++g) {
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, R, 0);
        }
    };

    // prologue: stages 0 .. S-1 in flight, then stage 0 resident
#pragma unroll
    for (int st = 0; st < S; ++st)
        if (st < nk) issue(st, kb + st * BK);
    wait_stages<Q, S - 1>(min(S - 1, nk - 1));
    __syncthreads();
    u32x4 f0a[MT], f0b[NT], f1a[MT], f1b[NT];
    load_half(0, 0, f0a, f0b);

    // stage kt: [read sub-step 1 | MFMAs of sub-step 0], then stage kt+1
    // resident + barrier (every wave has read all of stage kt, so its slot
    // takes stage kt+S), then [read sub-step 0 of kt+1 | MFMAs of sub-step 1].
    // The last stage re-reads itself (unused).
    for (int kt = 0; kt < nk; ++kt) {
        load_half(kt, 1, f1a, f1b);
        mma_half(f0a, f0b);
        const int left = nk - 2 - kt;
        wait_stages<Q, S - 1>(left < 0 ? 0 : left < S - 2 ? left : S - 2);   // stage kt+1 resident
        __syncthreads();
        if (kt + S < nk) issue(kt + S, kb + (kt + S) * BK);
        load_half(kt + 1 < nk ? kt + 1 : kt, 0, f0a, f0b);
        mma_half(f1a, f1b);
    }

    // epilogue: acc[i][t][e] is row m0 + wm*TM + 32i + 8(e/4) + 4kh + e%4, LDS B row wn*TN + 32t + r32
    int nrow[NT];
    bool nok[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) nrow[t] = wrow(wn * TN + 32 * t + r32, &nok[t]);
#pragma unroll
    for (int i = 0; i < MT; ++i) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int m = m0 + wm * TM + 32 * i + 8 * (e >> 2) + 4 * kh + (e & 3);
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
                    act[static_cast<size_t>(m) * p.ld_act + nrow[t]] = f32_to_bf16(swiglu_bf16(g, u));
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Full-line variant (K a multiple of 64): LDS rows of 64 elements (128 bytes),
// so each DMA instruction moves 8 whole 128-byte lines (the memory system
// serves full lines markedly faster than the half lines of the 64-byte-row
// ring).  Chunk c of row r sits at c ^ ((r / 2) % 8), which keeps the 32x32
// fragment reads free of bank conflicts.  A stage is 64 k (four 16-wide
// sub-steps).  The activation tile (re-read by every weight tile, so mostly
// L2 hits) and the weight tile (streamed from HBM) have rings of SA and SW
// stages (any pair; the kernels use SW >= SA): the slot of stage kt takes
// stage kt + SA (kt + SW) as soon as every wave has read all of stage kt, the
// activation DMA issued first so that the in-order load counter lets the
// weight stream stay in flight across the barrier (SW - 1 stages of
// lookahead for the weights).
// ---------------------------------------------------------------------------
// s_waitcnt vmcnt(<= n): rounded down to one of a few immediates (waiting for
// fewer outstanding loads than allowed is always safe)
__device__ __forceinline__ void wait_vm_atmost(int n) {
    if (n >= 48) wait_vm<48>();
    else if (n >= 32) wait_vm<32>();
    else if (n >= 24) wait_vm<24>();
    else if (n >= 16) wait_vm<16>();
    else if (n >= 12) wait_vm<12>();
    else if (n >= 8) wait_vm<8>();
    else if (n >= 6) wait_vm<6>();
    else if (n >= 4) wait_vm<4>();
    else if (n >= 2) wait_vm<2>();
    else wait_vm<0>();
}

template <int BM, int BN, int WM, int NW, int SA, int SW, int EPI, bool SPLIT>
__global__ void __launch_bounds__(64 * NW) gemm_dma128_kernel(GemmArgs p, int ksplit, int m_tiles, int n_tiles, int n0,
                                                              int gm, int xsplit) {
    constexpr int BK = 64, ROWB = 128;
    constexpr int WN = NW / WM;
    constexpr int TM = BM / WM, TN = BN / WN;
    constexpr int MT = TM / 32, NT = TN / 32;
    constexpr int ASTAGE = BM * ROWB, BSTAGE = BN * ROWB;
    constexpr int AQ = BM / (8 * NW), BQ = BN / (8 * NW);   // DMA instructions (8 rows each) per wave per stage
    static_assert(BM % (8 * NW) == 0 && BN % (8 * NW) == 0, "tile rows must fill whole DMA instructions");
    static_assert(TM % 32 == 0 && TN % 64 == 0, "wave tile must hold whole 32x32 tiles (and gate/up pairs)");
    static_assert(SA >= 2 && SW >= 2 && SA <= 6 && SW <= 6, "ring depths");
    constexpr int SMAX = SA > SW ? SA : SW;   // the prologue covers iterations -SMAX .. -1
    static_assert(SA * AQ + SW * BQ < 64, "vmcnt range (most loads ever in flight)");
    __shared__ __attribute__((aligned(1024))) uint8_t smem[SA * ASTAGE + SW * BSTAGE];

    const int w = blockIdx.x;
    const int xcd = w & 7, j = w >> 3;
    int m_tile, n_tile, split;
    if (xsplit) {
        // split-K over the XCDs: XCD x % 8 runs split 8y + x % 8 of every tile
        // (M tiles fastest), so its K range of the activations stays in its L2
        // and the M tiles of one weight tile run back to back
        split = static_cast<int>(blockIdx.y) * 8 + xcd;
        m_tile = j % m_tiles;
        n_tile = j / m_tiles;
        if (split * ksplit >= p.K || n_tile >= n_tiles) return;
    } else {
        const int ntx = (n_tiles + 7) >> 3;
        const int grp = j / (gm * ntx);
        const int rem = j - grp * gm * ntx;
        m_tile = grp * gm + rem % gm;
        n_tile = (rem / gm) * 8 + xcd;
        split = blockIdx.y;
        if (m_tile >= m_tiles || n_tile >= n_tiles) return;
    }

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WN, wn = wave % WN;
    const int r32 = lane & 31, kh = lane >> 5;
    const int M = p.M, Nw = p.Nw, K = p.K;
    const int m0 = m_tile * BM;

    auto wrow = [&](int b, bool* ok) -> int {
        if (EPI == EPI_SWIGLU) {
            const int wv = b / TN, u = b - wv * TN;
            const int c0 = n0 + n_tile * (BN / 2) + wv * (TN / 2);
            const int c = u < TN / 2 ? c0 + u : c0 + u - TN / 2;
            *ok = c < p.F;
            return u < TN / 2 ? c : p.F + c;
        } else {
            const int n = n0 + n_tile * BN + b;
            *ok = n < Nw;
            return n;
        }
    };

    const int kb = split * ksplit;
    const int ke = min(K, kb + ksplit);
    const int nk = (ke - kb) / BK;

    const uint16_t* A = static_cast<const uint16_t*>(p.A);
    const uint16_t* W = static_cast<const uint16_t*>(p.W);
    // DMA lane l of block g: row 8g + l/8, LDS chunk l%8 <- source chunk (l%8) ^ ((row/2)%8)
    const int lrow = lane >> 3;
    uint32_t aoff[AQ], boff[BQ];   // byte offsets (the launcher keeps them below 4 GiB)
#pragma unroll
    for (int q = 0; q < AQ; ++q) {
        const int g = wave * AQ + q;
        int m = m0 + 8 * g + lrow;
        m = m < M ? m : M - 1;
        const int ch = (lane & 7) ^ (((8 * g + lrow) >> 1) & 7);
        aoff[q] = 2u * (static_cast<uint32_t>(m) * static_cast<uint32_t>(p.lda) + 8u * ch);
    }
#pragma unroll
    for (int q = 0; q < BQ; ++q) {
        const int g = wave * BQ + q;
        bool ok;
        int n = wrow(8 * g + lrow, &ok);
        n = ok ? n : 0;
        const int ch = (lane & 7) ^ (((8 * g + lrow) >> 1) & 7);
        boff[q] = 2u * (static_cast<uint32_t>(n) * static_cast<uint32_t>(p.ldw) + 8u * ch);
    }
    uint8_t* const abuf = smem;
    uint8_t* const bbuf = smem + SA * ASTAGE;
    auto issue_a = [&](int stage) {
        uint8_t* base = abuf + (stage % SA) * ASTAGE;
        const uint8_t* src = reinterpret_cast<const uint8_t*>(A + kb + stage * BK);
#pragma unroll
        for (int q = 0; q < AQ; ++q) dma16_off(src, aoff[q], base + (wave * AQ + q) * 1024);
    };
    auto issue_w = [&](int stage) {
        uint8_t* base = bbuf + (stage % SW) * BSTAGE;
        const uint8_t* src = reinterpret_cast<const uint8_t*>(W + kb + stage * BK);
#pragma unroll
        for (int q = 0; q < BQ; ++q) dma16_off(src, boff[q], base + (wave * BQ + q) * 1024);
    };
    // Issue schedule: in (real or prologue) iteration i, A(i + SA) if in range,
    // then W(i + SW) if in range; the prologue is iterations -SMAX .. -1.
    auto issue_iter = [&](int i) {
        if (i + SA >= 0 && i + SA < nk) issue_a(i + SA);
        if (i + SW >= 0 && i + SW < nk) issue_w(i + SW);
    };
    // DMA instructions issued after the later of A(s), W(s), up to iteration `last`
    auto after_stage = [&](int s, int last) {
        const int ia = s - SA, iw = s - SW;   // issuing iterations
        int n = 0, i0;
        if (ia > iw) {                           // A(s) is issued after W(s): count W of its iteration
            i0 = ia;
            n += (i0 + SW >= 0 && i0 + SW < nk) ? BQ : 0;
        } else {                                 // same iteration, W(s) last
            i0 = iw;
        }
        for (int i = i0 + 1; i <= last; ++i)
            n += ((i + SA >= 0 && i + SA < nk) ? AQ : 0) + ((i + SW >= 0 && i + SW < nk) ? BQ : 0);
        return n;
    };

    f32x16 acc[MT][NT];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][t][e] = 0.f;

    // every fragment row is r32 plus a multiple of 32, so the swizzle depends on r32 only
    const int swz = (r32 >> 1) & 7;
    const uint32_t la = (wm * TM + r32) * ROWB, lb = (wn * TN + r32) * ROWB;
    auto load_sub = [&](int stage, int ks, u32x4 (&fa)[MT], u32x4 (&fb)[NT]) {
        const uint32_t ch = ((2 * ks + kh) ^ swz) << 4;
        const uint8_t* pa = abuf + (stage % SA) * ASTAGE + ch + la;
        const uint8_t* pb = bbuf + (stage % SW) * BSTAGE + ch + lb;
#pragma unroll
        for (int i = 0; i < MT; ++i) fa[i] = *reinterpret_cast<const u32x4*>(pa + 32 * i * ROWB);
#pragma unroll
        for (int t = 0; t < NT; ++t) fb[t] = *reinterpret_cast<const u32x4*>(pb + 32 * t * ROWB);
    };
    auto mma_sub = [&](const u32x4 (&fa)[MT], const u32x4 (&fb)[NT]) {
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int t = 0; t < NT; ++t)
                acc[i][t] = mfma32x32x16(as_bf16x8(fa[i]), as_bf16x8(fb[t]), acc[i][t]);
        constexpr int NRD = MT + NT, NMF = MT * NT;
        constexpr int R = NMF / NRD > 0 ? NMF / NRD : 1;
#pragma unroll
        for (int g = 0; g < NRD; ++g) {
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, R, 0);
        }
    };
    // The last sub-step of stage kt with the DMA issues of iteration kt,
    // A(kt + SA) then W(kt + SW) (both in range), spread between its MFMAs:
    // a wave held at a full load queue then still has matrix work queued.
    auto mma_sub_dma = [&](const u32x4 (&fa)[MT], const u32x4 (&fb)[NT], int kt) {
        constexpr int NMF = MT * NT, ND = AQ + BQ;
        const uint8_t* srca = reinterpret_cast<const uint8_t*>(A + kb + (kt + SA) * BK);
        const uint8_t* srcw = reinterpret_cast<const uint8_t*>(W + kb + (kt + SW) * BK);
        uint8_t* ldsa = abuf + ((kt + SA) % SA) * ASTAGE + wave * AQ * 1024;
        uint8_t* ldsw = bbuf + ((kt + SW) % SW) * BSTAGE + wave * BQ * 1024;
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int g = 0; g < NMF; ++g) {
            const int i = g / NT, t = g % NT;
            acc[i][t] = mfma32x32x16(as_bf16x8(fa[i]), as_bf16x8(fb[t]), acc[i][t]);
#pragma unroll
            for (int d = (ND * g) / NMF; d < (ND * (g + 1)) / NMF; ++d) {
                if (d < AQ) dma16_off(srca, aoff[d], ldsa + d * 1024);
                else dma16_off(srcw, boff[d - AQ], ldsw + (d - AQ) * 1024);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    for (int i = -SMAX; i < 0; ++i) issue_iter(i);
    if (nk > 0) wait_vm_atmost(after_stage(0, -1));
    __syncthreads();
    u32x4 f0a[MT], f0b[NT], f1a[MT], f1b[NT];
    load_sub(0, 0, f0a, f0b);

    // sub-steps 0..3 of stage kt alternate register sets; before the read of
    // stage kt+1 (under the MFMAs of sub-step 3) stage kt+1 must be resident
    // and every wave done with stage kt, whose slots then take A(kt+SA), W(kt+SW).
    int kt = 0;
    for (; kt + SMAX < nk; ++kt) {   // steady state: both issues in range
        load_sub(kt, 1, f1a, f1b);
        mma_sub(f0a, f0b);
        load_sub(kt, 2, f0a, f0b);
        mma_sub(f1a, f1b);
        load_sub(kt, 3, f1a, f1b);
        mma_sub(f0a, f0b);
        wait_vm_atmost(after_stage(kt + 1, kt - 1));   // stage kt+1 resident
        __syncthreads();
        load_sub(kt + 1, 0, f0a, f0b);
        mma_sub_dma(f1a, f1b, kt);
    }
    for (; kt < nk; ++kt) {
        load_sub(kt, 1, f1a, f1b);
        mma_sub(f0a, f0b);
        load_sub(kt, 2, f0a, f0b);
        mma_sub(f1a, f1b);
        load_sub(kt, 3, f1a, f1b);
        mma_sub(f0a, f0b);
        wait_vm_atmost(kt + 1 < nk ? after_stage(kt + 1, kt - 1) : 0);
        __syncthreads();
        issue_iter(kt);
        load_sub(kt + 1 < nk ? kt + 1 : kt, 0, f0a, f0b);
        mma_sub(f1a, f1b);
    }

    // epilogue: acc[i][t][e] is row m0 + wm*TM + 32i + 8(e/4) + 4kh + e%4, LDS B row wn*TN + 32t + r32
    int nrow[NT];
    bool nok[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) nrow[t] = wrow(wn * TN + 32 * t + r32, &nok[t]);
    // CHECKED: per-element row and column bounds (edge tiles); interior tiles
    // store without them
    auto store_tile = [&](auto checked) {
        constexpr bool CHECKED = decltype(checked)::value;
#pragma unroll
        for (int i = 0; i < MT; ++i) {
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int m = m0 + wm * TM + 32 * i + 8 * (e >> 2) + 4 * kh + (e & 3);
                if (CHECKED && m >= M) continue;
                if (SPLIT) {
                    float* dst = p.partial + (static_cast<size_t>(split) * M + m) * Nw;
#pragma unroll
                    for (int t = 0; t < NT; ++t)
                        if (!CHECKED || nok[t]) dst[nrow[t]] = acc[i][t][e];
                } else if (EPI == EPI_F32) {
#pragma unroll
                    for (int t = 0; t < NT; ++t)
                        if (!CHECKED || nok[t]) p.out_f32[static_cast<size_t>(m) * p.ldo + nrow[t]] = acc[i][t][e];
                } else if (EPI == EPI_RESID) {
#pragma unroll
                    for (int t = 0; t < NT; ++t)
                        if (!CHECKED || nok[t]) p.resid[static_cast<size_t>(m) * p.ldr + nrow[t]] += acc[i][t][e];
                } else {
                    uint16_t* act = static_cast<uint16_t*>(p.act);
#pragma unroll
                    for (int t = 0; t < NT / 2; ++t) {
                        if (CHECKED && !nok[t]) continue;
                        const float g = acc[i][t][e], u = acc[i][t + NT / 2][e];
                        act[static_cast<size_t>(m) * p.ld_act + nrow[t]] = f32_to_bf16(swiglu_bf16(g, u));
                    }
                }
            }
        }
    };
    bool inside = m0 + BM <= M;
#pragma unroll
    for (int t = 0; t < NT; ++t) inside = inside && nok[t];
    if (inside) store_tile(std::false_type{});
    else store_tile(std::true_type{});
}

template <int BM, int BN, int WM, int NW, int SA, int SW>
hipError_t launch_dma128(const GemmArgs& a, const GemmPlan& p, int n0, int n1, hipStream_t s) {
    const int m_tiles = (a.M + BM - 1) / BM;
    const int n_out = n1 - n0;
    const int bno = a.epi == EPI_SWIGLU ? BN / 2 : BN;
    const int n_tiles = (n_out + bno - 1) / bno;
    const int gm = m_tiles < 8 ? m_tiles : 8;
    const int ntx = (n_tiles + 7) / 8;
    const int groups = (m_tiles + gm - 1) / gm;
    // split-K counts that are multiples of 8: one split per XCD (see the kernel)
    const int xsplit = p.splits >= 8 && p.splits % 8 == 0;
    const dim3 grid = xsplit ? dim3(8 * m_tiles * n_tiles, p.splits / 8) : dim3(8 * ntx * groups * gm, p.splits);
    const dim3 block(64 * NW);
    if (p.splits > 1) {
        if (a.epi == EPI_SWIGLU)
            hipLaunchKernelGGL((gemm_dma128_kernel<BM, BN, WM, NW, SA, SW, EPI_SWIGLU, true>), grid, block, 0, s, a, p.ksplit, m_tiles, n_tiles, n0, gm, xsplit);
        else
            hipLaunchKernelGGL((gemm_dma128_kernel<BM, BN, WM, NW, SA, SW, EPI_F32, true>), grid, block, 0, s, a, p.ksplit, m_tiles, n_tiles, n0, gm, xsplit);
    } else if (a.epi == EPI_F32) {
        hipLaunchKernelGGL((gemm_dma128_kernel<BM, BN, WM, NW, SA, SW, EPI_F32, false>), grid, block, 0, s, a, p.ksplit, m_tiles, n_tiles, n0, gm, 0);
    } else if (a.epi == EPI_RESID) {
        hipLaunchKernelGGL((gemm_dma128_kernel<BM, BN, WM, NW, SA, SW, EPI_RESID, false>), grid, block, 0, s, a, p.ksplit, m_tiles, n_tiles, n0, gm, 0);
    } else {
        hipLaunchKernelGGL((gemm_dma128_kernel<BM, BN, WM, NW, SA, SW, EPI_SWIGLU, false>), grid, block, 0, s, a, p.ksplit, m_tiles, n_tiles, n0, gm, 0);
    }
    return hipGetLastError();
}

template <int BM, int BN, int WM, int NW, int S>
hipError_t launch_dma(const GemmArgs& a, const GemmPlan& p, int n0, int n1, hipStream_t s) {
    const int m_tiles = (a.M + BM - 1) / BM;
    const int n_out = n1 - n0;
    const int bno = a.epi == EPI_SWIGLU ? BN / 2 : BN;
    const int n_tiles = (n_out + bno - 1) / bno;
    const int gm = m_tiles < 8 ? m_tiles : 8;
    const int ntx = (n_tiles + 7) / 8;
    const int groups = (m_tiles + gm - 1) / gm;
    dim3 grid(8 * ntx * groups * gm, p.splits), block(64 * NW);
    if (p.splits > 1) {
        if (a.epi == EPI_SWIGLU)
            hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, WM, NW, S, EPI_SWIGLU, true>), grid, block, 0, s, a, p.ksplit, m_tiles, n_tiles, n0, gm);
        else
            hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, WM, NW, S, EPI_F32, true>), grid, block, 0, s, a, p.ksplit, m_tiles, n_tiles, n0, gm);
    } else if (a.epi == EPI_F32) {
        hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, WM, NW, S, EPI_F32, false>), grid, block, 0, s, a, p.ksplit, m_tiles, n_tiles, n0, gm);
    } else if (a.epi == EPI_RESID) {
        hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, WM, NW, S, EPI_RESID, false>), grid, block, 0, s, a, p.ksplit, m_tiles, n_tiles, n0, gm);
    } else {
        hipLaunchKernelGGL((gemm_dma_kernel<BM, BN, WM, NW, S, EPI_SWIGLU, false>), grid, block, 0, s, a, p.ksplit, m_tiles, n_tiles, n0, gm);
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

hipError_t launch_tile_variant(int variant, const GemmArgs& a, const GemmPlan& p, int n0, int n1, hipStream_t s) {
    switch (variant) {
        case kDmaVariant256x256: return launch_dma<256, 256, 2, 8, 5>(a, p, n0, n1, s);
        case kDmaVariant128x256: return launch_dma<128, 256, 2, 8, 6>(a, p, n0, n1, s);
        case kLineVariant256x256: return launch_dma128<256, 256, 2, 8, 2, 3>(a, p, n0, n1, s);
        case kLineVariant128x128: return launch_dma128<128, 128, 2, 4, 2, 3>(a, p, n0, n1, s);
        case kLineVariant128x256: return launch_dma128<128, 256, 2, 8, 3, 3>(a, p, n0, n1, s);
        case kLineVariant128x128Deep: return launch_dma128<128, 128, 2, 4, 4, 4>(a, p, n0, n1, s);
        default:   // register-staged tiles cover the whole output only
            if (n0 != 0) return hipErrorInvalidValue;
            return variant == kLdsVariant256 ? launch_tile<256, 128>(a, p, s) : launch_tile<128, 128>(a, p, s);
    }
}

}  // namespace

static hipError_t launch_segments(const GemmArgs& a, const GemmPlan& p, hipStream_t s) {
    const int n_out = a.epi == EPI_SWIGLU ? a.F : a.Nw;
    const int n_split = p.n_split > 0 && p.n_split < n_out ? p.n_split : n_out;
    hipError_t e = launch_tile_variant(p.variant, a, p, 0, n_split, s);
    if (e != hipSuccess || n_split == n_out) return e;
    GemmPlan q = p;
    q.splits = 1;
    q.ksplit = a.K;
    return launch_tile_variant(p.variant2, a, q, n_split, n_out, s);
}

// The tile kernels address A and W with 32-bit per-lane byte offsets: the
// weight rows must span less than 4 GiB, and larger M is run in row blocks
// that each do (split-K partials, laid out over the whole M, are never that
// large: their budget is far below).
hipError_t launch_gemm_bf16_lds(const GemmArgs& a, const GemmPlan& p, hipStream_t s) {
    if (a.M <= 0) return hipSuccess;
    constexpr uint64_t kOffLimit = 0xFFFFFFFFull;
    const uint64_t wrows = a.epi == EPI_SWIGLU ? 2ull * a.F : static_cast<uint64_t>(a.Nw);
    if (wrows * a.ldw * 2 > kOffLimit) return hipErrorInvalidValue;
    const uint64_t rows_max = kOffLimit / (2ull * a.lda) / 256 * 256;
    if (static_cast<uint64_t>(a.M) <= rows_max) return launch_segments(a, p, s);
    if (p.splits > 1 || rows_max == 0) return hipErrorInvalidValue;
    for (int m0 = 0; m0 < a.M; m0 += static_cast<int>(rows_max)) {
        GemmArgs b = a;
        b.M = static_cast<int>(std::min<uint64_t>(rows_max, static_cast<uint64_t>(a.M - m0)));
        b.A = static_cast<const uint16_t*>(a.A) + static_cast<size_t>(m0) * a.lda;
        if (b.out_f32) b.out_f32 += static_cast<size_t>(m0) * a.ldo;
        if (b.resid) b.resid += static_cast<size_t>(m0) * a.ldr;
        if (b.act) b.act = static_cast<uint16_t*>(a.act) + static_cast<size_t>(m0) * a.ld_act;
        const hipError_t e = launch_segments(b, p, s);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace rl
