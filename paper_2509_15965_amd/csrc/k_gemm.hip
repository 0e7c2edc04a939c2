// k_gemm.hip -- Y = X . W^T for the projections, MLP and LM head.
//
// bf16: MFMA 16x16x32 tiles fed straight from global memory.  A lane loads
// 16 contiguous bytes of one row (8 k values) per 32-wide k group, so 16
// lanes sharing a k group read 16 rows and the 4 k groups of a wave read 64
// contiguous bytes of every row: weight rows stream from HBM in full 128-byte
// lines across the two MFMAs of a 64-wide k step, each weight byte read once
// per workgroup row.  Small batches (M <= 64) use one 16/32/64-row M tile per
// workgroup and split K across workgroups when the weight alone cannot fill
// the 256 CUs; fp32 partials are then summed in a fixed order by
// splitk_reduce (deterministic).  Larger batches go to the LDS-tiled kernel
// (k_gemm_lds.hip).
//
// fp32: a plain LDS-tiled VALU kernel (the tiny fp32 decoder only).
#include "rl_decode.h"
#include "rl_device.h"
#include "rl_internal.h"

namespace rl {

const GemmShape kGemmShapes[kNumGemmShapes] = {
    {1, 4, 1, 4},   // M <= 16 : 16 x 256 weight rows per workgroup
    {2, 4, 1, 4},   // M <= 32 : 32 x 256
    {4, 4, 1, 4},   // M <= 64 : 64 x 256
};

static int ceil_div(int a, int b) { return (a + b - 1) / b; }

namespace {

// Tile kernels of the batched (M > 64) path for the planner's cost model:
// tile shape, workgroups resident per CU, and the measured time of one
// round (every CU busy) per 1024 k, in microseconds.  A lone 128 x 128
// workgroup on a CU runs faster than a co-resident pair (t_alone).
struct TileKernel { int variant, BM, BN, per_cu; double t_round, t_alone; };
constexpr TileKernel kLineTiles[] = {   // ties go to the earlier entry (weights not cache resident)
    {kLineVariant256x256, 256, 256, 1, 31.0, 31.0},
    {kLineVariant128x128, 128, 128, 2, 20.3, 15.0},
    {kLineVariant128x256, 128, 256, 1, 19.5, 19.5},
    {kLineVariant128x128Deep, 128, 128, 1, 12.0, 12.0},
};
constexpr int kCUs = 256;

struct Cost { double us; };

double rounds_us(const TileKernel& t, long tiles, double kfrac) {
    const long per_cu = (tiles + kCUs - 1) / kCUs;
    if (t.per_cu == 1) return per_cu * t.t_round * kfrac;
    return (per_cu / 2) * t.t_round * kfrac + (per_cu % 2) * t.t_alone * kfrac;
}

long tiles_of(const TileKernel& t, int M, int n_cols, int epi) {
    const int bno = epi == EPI_SWIGLU ? t.BN / 2 : t.BN;
    return static_cast<long>(ceil_div(M, t.BM)) * ceil_div(n_cols, bno);
}

}  // namespace

// Direct-load kernel plan for M <= 64 (its own split-K heuristic: split until
// about 1024 workgroups stream the weight).
GemmPlan plan_direct(int M, int Nw, int K, int epi, int F) {
    GemmPlan p{};
    const int n_out = epi == EPI_SWIGLU ? F : Nw;
    p.variant = M <= 16 ? 0 : M <= 32 ? 1 : 2;
    const GemmShape& s = kGemmShapes[p.variant];
    const int BM = 16 * s.MT * s.WR;
    const int BNw = 16 * s.NT * s.WC;
    const int BNo = epi == EPI_SWIGLU ? BNw / 2 : BNw;
    p.grid_x = ceil_div(n_out, BNo);
    p.grid_y = ceil_div(M, BM);
    const long tiles = static_cast<long>(p.grid_x) * p.grid_y;
    // smallest K slice per split: partial sums cost 4*M bytes per output for
    // every 2*slice bytes of weight read, so tiny batches can split finely
    const int min_ks = M <= 16 ? 128 : M <= 32 ? 256 : 512;
    int S = 1;
    while (tiles * S * 2 <= 1024 && ceil_div(K, 2 * S) >= min_ks &&
           static_cast<size_t>(2 * S) * M * Nw <= kPartCapFloats && 2 * S <= kMaxSplits)
        S *= 2;
    const int ks = ceil_div(ceil_div(K, S), 64) * 64;
    p.ksplit = ks;
    p.splits = ceil_div(K, ks);
    return p;
}

// Plan of one bf16 GEMM: the cheapest of
//  (a) the direct-load kernel (M <= 16, or M <= 64 when K % 64 != 0) or the
//      GEMV-shaped kernel (M <= 32, no split-K),
//  (b) one LDS tile kernel with split-K s (partials summed by splitk_reduce),
//  (c) 256 x 256 tiles for whole rounds plus a smaller tile kernel for the
//      remaining output columns,
// under a cost model (microseconds): rounds x measured round time, partial-sum
// and output traffic, a fixed pipeline cost for tile kernels on small batches,
// and a floor at the HBM rate for the weight stream.  K % 64 != 0 (not used by
// the decoder shapes) falls back to the 64-byte-row / register-staged tiles.
GemmPlan plan_gemm_bf16(int M, int Nw, int K, int epi, int F) {
    const int n_out = epi == EPI_SWIGLU ? F : Nw;
    const double wbytes = 2.0 * Nw * K;
    const double floor_us = wbytes / 5.2e6;
    const double out_us = (epi == EPI_F32 ? 4.0 : epi == EPI_RESID ? 8.0 : 2.0) * M * n_out / 4.0e6;
    auto reduce_us = [&](int s) { return s > 1 ? 8.0 * s * M * static_cast<double>(Nw) / 3.0e6 + 4.0 : 0.0; };

    GemmPlan best_p{};
    double best = 1e30;
    if (M <= 16 || (M <= 64 && K % 64 != 0)) {
        best_p = plan_direct(M, Nw, K, epi, F);
        best = wbytes / 3.6e6 * (1.0 + M / 60.0) + reduce_us(best_p.splits) + 2.0;
    }
    if (M <= 32 && K % 64 == 0) {
        // GEMV-shaped kernel: a CU streams ~24 GB/s of its workgroups' 16
        // weight rows; each workgroup also reads the M activation rows from L2
        // (measured to cost ~0.65 of the same bytes of weight)
        const double wg_bytes = 16.0 * K * 2.0 * (1.0 + 0.65 * M / 16.0);
        const long wgs = epi == EPI_SWIGLU ? ceil_div(F, 8) : ceil_div(Nw, 16);
        const long per_cu = (wgs + kCUs - 1) / kCUs;
        const double us = per_cu * wg_bytes / 24.0e3 + 3.0 + out_us;
        if (us < best * 0.98) {
            best = us;
            best_p = GemmPlan{};
            best_p.variant = kGemvVariant; best_p.splits = 1; best_p.ksplit = K;
        }
    }
    if (K % 64 != 0) {
        if (M <= 64) return best_p;
        GemmPlan p{};
        int BM, BN;
        if (K % 32 == 0) {
            p.variant = M > 128 ? kDmaVariant256x256 : kDmaVariant128x256; BM = M > 128 ? 256 : 128; BN = 256;
        } else {
            p.variant = M > 128 ? kLdsVariant256 : kLdsVariant128; BM = M > 128 ? 256 : 128; BN = 128;
        }
        const int bno = epi == EPI_SWIGLU ? BN / 2 : BN;
        p.grid_x = ceil_div(n_out, bno);
        p.grid_y = ceil_div(M, BM);
        const long tiles = static_cast<long>(p.grid_x) * p.grid_y;
        int S = 1;
        while (tiles * S * 2 <= 240 && ceil_div(K, 2 * S) >= 256 &&
               static_cast<size_t>(2 * S) * M * Nw <= kPartCapFloats && 2 * S <= kMaxSplits)
            S *= 2;
        const int ks = ceil_div(ceil_div(K, S), 64) * 64;
        p.ksplit = ks;
        p.splits = ceil_div(K, ks);
        return p;
    }
    const double fixed = M <= 64 ? 5.0 : 0.0;
    for (const TileKernel& t : kLineTiles) {
        const long tiles = tiles_of(t, M, n_out, epi);
        for (int s = 1; s <= kMaxSplits; s *= 2) {
            const int ks = ceil_div(ceil_div(K, s), 64) * 64;
            if (s > 1 && (ceil_div(K, ks) != s || ks < 256 || static_cast<size_t>(s) * M * Nw > kPartCapFloats))
                break;
            double us = rounds_us(t, tiles * s, ks / 1024.0);
            us = (us > floor_us ? us : floor_us) + out_us + reduce_us(s) + fixed;
            if (us < best * 0.98) {
                best = us;
                best_p = GemmPlan{};
                best_p.variant = t.variant; best_p.splits = s; best_p.ksplit = ks;
            }
        }
    }
    // whole rounds of 256 x 256 tiles, then the rest of the columns
    const TileKernel& big = kLineTiles[0];
    const long big_tiles = tiles_of(big, M, n_out, epi);
    const int m_tiles = ceil_div(M, big.BM);
    const int bno = epi == EPI_SWIGLU ? big.BN / 2 : big.BN;
    const long full_cols = (big_tiles / kCUs) * kCUs / m_tiles;   // n tiles of whole rounds
    if (full_cols > 0 && full_cols * bno < n_out) {
        const int n_split = static_cast<int>(full_cols * bno);
        const double kf = K / 1024.0;
        for (int v = 1; v < 4; ++v) {
            const TileKernel& t = kLineTiles[v];
            double us = rounds_us(big, full_cols * m_tiles, kf) +
                        rounds_us(t, tiles_of(t, M, n_out - n_split, epi), kf);
            us = (us > floor_us ? us : floor_us) + out_us + 4.0 + fixed;
            if (us < best * 0.98) {
                best = us;
                best_p = GemmPlan{};
                best_p.variant = big.variant; best_p.splits = 1; best_p.ksplit = K;
                best_p.n_split = n_split; best_p.variant2 = t.variant;
            }
        }
    }
    return best_p;
}

// Every plan of the cost model's search space for this GEMM, its own choice
// first: the direct-load kernel (M <= 64) at split counts 1..16, the
// GEMV-shaped kernel (M <= 32), and from 16 rows each batched tile kernel at
// every split count the cost model prices (powers of two, slices of at least
// 256 k, partials within budget) and the two-segment launches of whole
// 256 x 256 rounds plus a smaller tile kernel (below 16 rows the tiles are
// mostly empty rows and were never faster than the GEMV or direct kernels).
// K % 64 != 0 has no alternatives.  Returns the count written (at most cap).
constexpr int kMinTileCandidateRows = 16;
int plan_gemm_candidates(int M, int Nw, int K, int epi, int F, GemmPlan* out, int cap) {
    int n = 0;
    auto same = [](const GemmPlan& a, const GemmPlan& b) {
        return a.variant == b.variant && a.splits == b.splits && a.ksplit == b.ksplit && a.n_split == b.n_split &&
               a.variant2 == b.variant2 && a.grid_x == b.grid_x && a.grid_y == b.grid_y;
    };
    auto add = [&](const GemmPlan& p) {
        for (int i = 0; i < n; ++i)
            if (same(out[i], p)) return;
        if (n < cap) out[n++] = p;
    };
    add(plan_gemm_bf16(M, Nw, K, epi, F));
    if (K % 64 != 0) return n;
    const int n_out = epi == EPI_SWIGLU ? F : Nw;
    if (M <= 64) {
        for (int s = 1; s <= 16; s *= 2) {
            GemmPlan p = plan_direct(M, Nw, K, epi, F);
            const int ks = ceil_div(ceil_div(K, s), 64) * 64;
            if (static_cast<size_t>(ceil_div(K, ks)) * M * Nw > kPartCapFloats) break;
            p.ksplit = ks;
            p.splits = ceil_div(K, ks);
            add(p);
        }
    }
    if (M <= 32) {
        GemmPlan p{};
        p.variant = kGemvVariant; p.splits = 1; p.ksplit = K;
        add(p);
    }
    if (M <= 64) {
        // the wide GEMV at 1..8 K slices of at least 256 (64 per wave)
        for (int sp = 1; sp <= 8; sp *= 2) {
            GemmPlan p{};
            p.variant = kGemvWideVariant;
            p.ksplit = ceil_div(ceil_div(K, sp), 64) * 64;
            p.splits = ceil_div(K, p.ksplit);
            if (sp > 1 && (p.ksplit < 256 || static_cast<size_t>(p.splits) * M * Nw > kPartCapFloats)) break;
            add(p);
        }
    }
    if (M < kMinTileCandidateRows) return n;
    for (const TileKernel& t : kLineTiles) {
        for (int s = 1; s <= kMaxSplits; s *= 2) {
            const int ks = ceil_div(ceil_div(K, s), 64) * 64;
            if (s > 1 && (ceil_div(K, ks) != s || ks < 256 || static_cast<size_t>(s) * M * Nw > kPartCapFloats))
                break;
            GemmPlan p{};
            p.variant = t.variant; p.splits = s; p.ksplit = ks;
            add(p);
        }
    }
    const TileKernel& big = kLineTiles[0];
    const long big_tiles = tiles_of(big, M, n_out, epi);
    const int m_tiles = ceil_div(M, big.BM);
    const int bno = epi == EPI_SWIGLU ? big.BN / 2 : big.BN;
    const long full_cols = (big_tiles / kCUs) * kCUs / m_tiles;
    if (full_cols > 0 && full_cols * bno < n_out) {
        for (int v = 1; v < 4; ++v) {
            GemmPlan p{};
            p.variant = big.variant; p.splits = 1; p.ksplit = K;
            p.n_split = static_cast<int>(full_cols * bno); p.variant2 = kLineTiles[v].variant;
            add(p);
        }
    }
    return n;
}

// The RL_OPT_GEMM_PLAN code of a plan (0 when it has none).
int64_t gemm_plan_code_of(const GemmPlan& p) {
    auto code = [](int v) -> int64_t {
        switch (v) {
            case kLineVariant256x256: return RL_GEMM_T256;
            case kLineVariant128x256: return RL_GEMM_T128X256;
            case kLineVariant128x128: return RL_GEMM_T128;
            case kLineVariant128x128Deep: return RL_GEMM_T128_DEEP;
            case kGemvVariant: return RL_GEMM_GEMV;
            case kGemvWideVariant: return RL_GEMM_GEMV_WIDE;
            default: return v >= 0 && v < kNumGemmShapes ? RL_GEMM_DIRECT : 0;
        }
    };
    const int64_t k1 = code(p.variant);
    if (k1 == 0) return 0;
    const int64_t s = p.splits > 1 ? p.splits : 0;
    const int64_t k2 = p.n_split > 0 ? code(p.variant2) : 0;
    return k1 | (s << 8) | (k2 << 16);
}

bool plan_gemm_forced(int M, int Nw, int K, int epi, int F, int64_t code, GemmPlan* out) {
    const int k1 = static_cast<int>(code & 0xff), s = static_cast<int>((code >> 8) & 0xff);
    const int k2 = static_cast<int>((code >> 16) & 0xff);
    const int n_out = epi == EPI_SWIGLU ? F : Nw;
    auto tile = [](int k) {
        switch (k) {
            case RL_GEMM_T256: return kLineVariant256x256;
            case RL_GEMM_T128X256: return kLineVariant128x256;
            case RL_GEMM_T128: return kLineVariant128x128;
            case RL_GEMM_T128_DEEP: return kLineVariant128x128Deep;
            default: return -1;
        }
    };
    auto out_width = [&](int v) {
        const int bn = v == kLineVariant128x128 || v == kLineVariant128x128Deep ? 128 : 256;
        return epi == EPI_SWIGLU ? bn / 2 : bn;
    };
    if (s > kMaxSplits) return false;
    GemmPlan p{};
    if (k1 == RL_GEMM_DIRECT) {
        if (M > 64 || k2 != 0) return false;
        p = plan_direct(M, Nw, K, epi, F);
        if (s > 1) {
            const int ks = ceil_div(ceil_div(K, s), 64) * 64;
            if (static_cast<size_t>(ceil_div(K, ks)) * M * Nw > kPartCapFloats) return false;
            p.ksplit = ks;
            p.splits = ceil_div(K, ks);
        } else if (s == 1) {
            p.ksplit = K;
            p.splits = 1;
        }
        *out = p;
        return true;
    }
    if (k1 == RL_GEMM_GEMV) {
        if (M > 32 || K % 64 != 0 || k2 != 0) return false;
        p.variant = kGemvVariant; p.splits = 1; p.ksplit = K;
        *out = p;
        return true;
    }
    if (k1 == RL_GEMM_GEMV_WIDE) {
        if (M > 64 || K % 64 != 0 || k2 != 0) return false;
        p.variant = kGemvWideVariant;
        p.ksplit = s > 1 ? ceil_div(ceil_div(K, s), 64) * 64 : K;
        p.splits = ceil_div(K, p.ksplit);
        if (p.splits > 1 && static_cast<size_t>(p.splits) * M * Nw > kPartCapFloats) return false;
        *out = p;
        return true;
    }
    const int v1 = tile(k1);
    if (v1 < 0 || K % 64 != 0) return false;
    p.variant = v1;
    p.splits = 1;
    p.ksplit = K;
    if (k2 != 0) {
        const int v2 = tile(k2);
        if (v2 < 0) return false;
        const int w = out_width(v1);
        const int n_split = (n_out / 2) / w * w;
        if (n_split <= 0) return false;
        p.n_split = n_split;
        p.variant2 = v2;
    } else if (s > 1) {
        const int ks = ceil_div(ceil_div(K, s), 64) * 64;
        const int splits = ceil_div(K, ks);
        if (static_cast<size_t>(splits) * M * Nw > kPartCapFloats) return false;
        p.ksplit = ks;
        p.splits = splits;
    }
    *out = p;
    return true;
}

// ---------------------------------------------------------------------------
// bf16 MFMA kernel
// ---------------------------------------------------------------------------
template <int MT, int NT, int WR, int WC, int EPI, bool SPLIT>
__global__ void __launch_bounds__(256) gemm_bf16_kernel(GemmArgs p, int ksplit) {
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wr = wave / WC, wc = wave % WC;
    const int r16 = lane & 15, kq = lane >> 4;
    const int M = p.M, Nw = p.Nw, K = p.K;

    const int m_base = (blockIdx.y * WR + wr) * 16 * MT;
    // weight row of tile t (the SwiGLU wave takes matching gate and up tiles)
    int wrow[NT];
    if (EPI == EPI_SWIGLU) {
        const int c0 = (blockIdx.x * WC + wc) * 16 * (NT / 2);
#pragma unroll
        for (int t = 0; t < NT; ++t)
            wrow[t] = t < NT / 2 ? c0 + 16 * t : p.F + c0 + 16 * (t - NT / 2);
    } else {
        const int n0 = (blockIdx.x * WC + wc) * 16 * NT;
#pragma unroll
        for (int t = 0; t < NT; ++t) wrow[t] = n0 + 16 * t;
    }

    const int kb = blockIdx.z * ksplit;
    const int ke = min(K, kb + ksplit);

    const uint16_t* A = static_cast<const uint16_t*>(p.A);
    const uint16_t* W = static_cast<const uint16_t*>(p.W);
    const uint16_t* ap[MT];
    bool aok[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i) {
        const int m = m_base + 16 * i + r16;
        aok[i] = m < M;
        ap[i] = A + static_cast<size_t>(aok[i] ? m : 0) * p.lda + 8 * kq;
    }
    const uint16_t* wp[NT];
    bool wok[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int n = wrow[t] + r16;
        bool ok = n < Nw;
        if (EPI == EPI_SWIGLU) {
            const int c = t < NT / 2 ? n : n - p.F;
            ok = c < p.F;
        }
        wok[t] = ok;
        wp[t] = W + static_cast<size_t>(ok ? n : 0) * p.ldw + 8 * kq;
    }

    f32x4 acc[MT][NT];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[i][t] = f32x4{0.f, 0.f, 0.f, 0.f};

    const u32x4 zero = {0u, 0u, 0u, 0u};
    u32x4 a_cur[MT][2], b_cur[NT][2];
    auto load = [&](u32x4 (&a)[MT][2], u32x4 (&b)[NT][2], int k0) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int kk = k0 + 32 * j + 8 * kq;
            const bool kok = kk < ke;
#pragma unroll
            for (int i = 0; i < MT; ++i) a[i][j] = (aok[i] && kok) ? ld16(ap[i] + k0 + 32 * j) : zero;
#pragma unroll
            for (int t = 0; t < NT; ++t) b[t][j] = (wok[t] && kok) ? ld16(wp[t] + k0 + 32 * j) : zero;
        }
    };

    if (kb < ke) load(a_cur, b_cur, kb);
    for (int k0 = kb; k0 < ke; k0 += 64) {
        u32x4 a_nxt[MT][2], b_nxt[NT][2];
        const bool more = k0 + 64 < ke;
        if (more) load(a_nxt, b_nxt, k0 + 64);
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int i = 0; i < MT; ++i)
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    acc[i][t] = mfma16x16x32(as_bf16x8(a_cur[i][j]), as_bf16x8(b_cur[t][j]), acc[i][t]);
        if (more) {
#pragma unroll
            for (int j = 0; j < 2; ++j) {
#pragma unroll
                for (int i = 0; i < MT; ++i) a_cur[i][j] = a_nxt[i][j];
#pragma unroll
                for (int t = 0; t < NT; ++t) b_cur[t][j] = b_nxt[t][j];
            }
        }
    }

    // epilogue: lane holds rows m_base + 16 i + 4 kq + e, weight row wrow[t] + r16
#pragma unroll
    for (int i = 0; i < MT; ++i) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int m = m_base + 16 * i + 4 * kq + e;
            if (m >= M) continue;
            if (SPLIT) {
                float* dst = p.partial + (static_cast<size_t>(blockIdx.z) * M + m) * Nw;
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    const int n = wrow[t] + r16;
                    if (wok[t]) dst[n] = acc[i][t][e];
                }
            } else if (EPI == EPI_F32) {
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    const int n = wrow[t] + r16;
                    if (wok[t]) p.out_f32[static_cast<size_t>(m) * p.ldo + n] = acc[i][t][e];
                }
            } else if (EPI == EPI_RESID) {
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    const int n = wrow[t] + r16;
                    if (wok[t]) p.resid[static_cast<size_t>(m) * p.ldr + n] += acc[i][t][e];
                }
            } else {  // EPI_SWIGLU
                uint16_t* act = static_cast<uint16_t*>(p.act);
#pragma unroll
                for (int t = 0; t < NT / 2; ++t) {
                    const int c = wrow[t] + r16;
                    if (!wok[t]) continue;
                    const float g = acc[i][t][e], u = acc[i][t + NT / 2][e];
                    act[static_cast<size_t>(m) * p.ld_act + c] = f32_to_bf16(swiglu_bf16(g, u));
                }
            }
        }
    }
}

template <int MT, int NT, int WR, int WC>
static hipError_t launch_shape(const GemmArgs& a, const GemmPlan& p, hipStream_t s) {
    dim3 grid(p.grid_x, p.grid_y, p.splits), block(256);
    if (p.splits > 1) {
        if (a.epi == EPI_SWIGLU)
            hipLaunchKernelGGL((gemm_bf16_kernel<MT, NT, WR, WC, EPI_SWIGLU, true>), grid, block, 0, s, a, p.ksplit);
        else
            hipLaunchKernelGGL((gemm_bf16_kernel<MT, NT, WR, WC, EPI_F32, true>), grid, block, 0, s, a, p.ksplit);
    } else if (a.epi == EPI_F32) {
        hipLaunchKernelGGL((gemm_bf16_kernel<MT, NT, WR, WC, EPI_F32, false>), grid, block, 0, s, a, p.ksplit);
    } else if (a.epi == EPI_RESID) {
        hipLaunchKernelGGL((gemm_bf16_kernel<MT, NT, WR, WC, EPI_RESID, false>), grid, block, 0, s, a, p.ksplit);
    } else {
        hipLaunchKernelGGL((gemm_bf16_kernel<MT, NT, WR, WC, EPI_SWIGLU, false>), grid, block, 0, s, a, p.ksplit);
    }
    return hipGetLastError();
}

hipError_t launch_gemv(const GemmArgs& a, hipStream_t s);
hipError_t launch_gemv_wide(const GemmArgs& a, const GemmPlan& p, hipStream_t s);

hipError_t launch_gemm_bf16(const GemmArgs& a, const GemmPlan& p, hipStream_t s) {
    if (a.M <= 0) return hipSuccess;
    switch (p.variant) {
        case 0: return launch_shape<1, 4, 1, 4>(a, p, s);
        case 1: return launch_shape<2, 4, 1, 4>(a, p, s);
        case 2: return launch_shape<4, 4, 1, 4>(a, p, s);
        case kGemvVariant: return launch_gemv(a, s);
        case kGemvWideVariant: return launch_gemv_wide(a, p, s);
        default: return launch_gemm_bf16_lds(a, p, s);
    }
}

// ---------------------------------------------------------------------------
// GEMV-shaped kernel for M <= 32: one workgroup (8 waves) owns 16 weight rows
// (SwiGLU: 8 gate rows and the matching 8 up rows) and the whole K.  Wave w
// takes the w-th eighth of K, streams its weight and activation fragments
// straight from global memory (16-byte loads, four 64-wide k blocks in flight
// per wave) into 16x16x32 MFMAs, and the eight partial 16x16 tiles are summed
// through LDS in wave order (deterministic) before the epilogue.  No split-K
// partials and no reduction kernel.
// ---------------------------------------------------------------------------
template <int MR, int EPI>
__global__ void __launch_bounds__(512) gemv_kernel(GemmArgs p, int kw) {
    constexpr int U = 4;   // 64-wide k blocks per batch of loads
    __shared__ f32x4 red[8][MR][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r16 = lane & 15, kq = lane >> 4;
    const int M = p.M, K = p.K;

    int n;
    bool ok;
    if (EPI == EPI_SWIGLU) {
        const int c = blockIdx.x * 8 + (r16 & 7);
        ok = c < p.F;
        n = r16 < 8 ? c : p.F + c;
    } else {
        n = blockIdx.x * 16 + r16;
        ok = n < p.Nw;
    }
    const uint16_t* wp = static_cast<const uint16_t*>(p.W) + static_cast<size_t>(ok ? n : 0) * p.ldw + 8 * kq;
    const uint16_t* ap[MR];
    bool aok[MR];
#pragma unroll
    for (int i = 0; i < MR; ++i) {
        const int m = 16 * i + r16;
        aok[i] = m < M;
        ap[i] = static_cast<const uint16_t*>(p.A) + static_cast<size_t>(aok[i] ? m : 0) * p.lda + 8 * kq;
    }
    const int kb = wave * kw;
    const int ke = min(K, kb + kw);

    f32x4 acc[MR];
#pragma unroll
    for (int i = 0; i < MR; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    const u32x4 zero = {0u, 0u, 0u, 0u};
    for (int k0 = kb; k0 < ke; k0 += 64 * U) {
        u32x4 wf[U][2], af[U][2][MR];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int kk = k0 + 64 * u + 32 * j;
                const bool kok = kk + 8 * kq < ke;
                wf[u][j] = (ok && kok) ? ld16(wp + kk) : zero;
#pragma unroll
                for (int i = 0; i < MR; ++i) af[u][j][i] = (aok[i] && kok) ? ld16(ap[i] + kk) : zero;
            }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int i = 0; i < MR; ++i)
                    acc[i] = mfma16x16x32(as_bf16x8(af[u][j][i]), as_bf16x8(wf[u][j]), acc[i]);
    }
#pragma unroll
    for (int i = 0; i < MR; ++i) red[wave][i][lane] = acc[i];
    __syncthreads();
    if (wave >= MR) return;
    // wave i sums A tile i over the 8 waves in order; lane holds D[4 kq + e][r16]
    f32x4 v = red[0][wave][lane];
#pragma unroll
    for (int w = 1; w < 8; ++w) v += red[w][wave][lane];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int m = 16 * wave + 4 * kq + e;
        const float val = v[e];
        if (EPI == EPI_SWIGLU) {
            const float up = __shfl(val, (lane & ~15) | ((r16 + 8) & 15), 64);
            if (r16 < 8 && ok && m < M) {
                static_cast<uint16_t*>(p.act)[static_cast<size_t>(m) * p.ld_act + n] = f32_to_bf16(swiglu_bf16(val, up));
            }
        } else if (ok && m < M) {
            if (EPI == EPI_F32) p.out_f32[static_cast<size_t>(m) * p.ldo + n] = val;
            else p.resid[static_cast<size_t>(m) * p.ldr + n] += val;
        }
    }
}

hipError_t launch_gemv(const GemmArgs& a, hipStream_t s) {
    const int kw = ceil_div(ceil_div(a.K, 8), 64) * 64;
    const int blocks = a.epi == EPI_SWIGLU ? ceil_div(a.F, 8) : ceil_div(a.Nw, 16);
    dim3 grid(blocks), block(512);
#define RL_GV(MR)                                                                                        \
    do {                                                                                                 \
        if (a.epi == EPI_F32) hipLaunchKernelGGL((gemv_kernel<MR, EPI_F32>), grid, block, 0, s, a, kw);   \
        else if (a.epi == EPI_RESID) hipLaunchKernelGGL((gemv_kernel<MR, EPI_RESID>), grid, block, 0, s, a, kw); \
        else hipLaunchKernelGGL((gemv_kernel<MR, EPI_SWIGLU>), grid, block, 0, s, a, kw);                 \
    } while (0)
    if (a.M <= 16) RL_GV(1);
    else if (a.M <= 32) RL_GV(2);
    else return hipErrorInvalidValue;
#undef RL_GV
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Wide GEMV-shaped kernel for M <= 64: one workgroup (4 waves) owns 64 weight
// rows (SwiGLU: 32 gate rows and the matching 32 up rows) and one K slice
// (blockIdx.y; the whole K without split-K); wave w takes the w-th quarter
// of the slice.  Every activation fragment a wave loads feeds four 16-row
// weight groups, so a workgroup re-reads the M activation rows once per 64
// weight rows instead of once per 16.  The four partial tiles are summed
// through LDS in wave order (deterministic); split-K slices land in the
// partials buffer [splits][M][Nw] like the other kernels' slices.
// ---------------------------------------------------------------------------
template <int MR, int EPI, bool SPLIT>
__global__ void __launch_bounds__(256) gemv_wide_kernel(GemmArgs p, int ksplit, int kw) {
    constexpr int NT = 4;   // 16-row weight groups per workgroup
    constexpr int U = 2;    // 64-wide k blocks per batch of loads
    __shared__ f32x4 red[4][MR * NT][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r16 = lane & 15, kq = lane >> 4;
    const int M = p.M;

    int n[NT];
    bool ok[NT];
    const uint16_t* wp[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        if (EPI == EPI_SWIGLU) {
            const int c = (blockIdx.x * NT + t) * 8 + (r16 & 7);
            ok[t] = c < p.F;
            n[t] = r16 < 8 ? c : p.F + c;
        } else {
            n[t] = (blockIdx.x * NT + t) * 16 + r16;
            ok[t] = n[t] < p.Nw;
        }
        wp[t] = static_cast<const uint16_t*>(p.W) + static_cast<size_t>(ok[t] ? n[t] : 0) * p.ldw + 8 * kq;
    }
    const uint16_t* ap[MR];
    bool aok[MR];
#pragma unroll
    for (int i = 0; i < MR; ++i) {
        const int m = 16 * i + r16;
        aok[i] = m < M;
        ap[i] = static_cast<const uint16_t*>(p.A) + static_cast<size_t>(aok[i] ? m : 0) * p.lda + 8 * kq;
    }
    const int ks0 = blockIdx.y * ksplit;
    const int ks1 = min(p.K, ks0 + ksplit);
    const int kb = ks0 + wave * kw;
    const int ke = min(ks1, kb + kw);

    f32x4 acc[MR][NT];
#pragma unroll
    for (int i = 0; i < MR; ++i)
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[i][t] = f32x4{0.f, 0.f, 0.f, 0.f};
    const u32x4 zero = {0u, 0u, 0u, 0u};
    for (int k0 = kb; k0 < ke; k0 += 64 * U) {
        u32x4 wf[U][2][NT], af[U][2][MR];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int kk = k0 + 64 * u + 32 * j;
                const bool kok = kk + 8 * kq < ke;
#pragma unroll
                for (int t = 0; t < NT; ++t) wf[u][j][t] = (ok[t] && kok) ? ld16(wp[t] + kk) : zero;
#pragma unroll
                for (int i = 0; i < MR; ++i) af[u][j][i] = (aok[i] && kok) ? ld16(ap[i] + kk) : zero;
            }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int i = 0; i < MR; ++i)
#pragma unroll
                    for (int t = 0; t < NT; ++t)
                        acc[i][t] = mfma16x16x32(as_bf16x8(af[u][j][i]), as_bf16x8(wf[u][j][t]), acc[i][t]);
    }
#pragma unroll
    for (int i = 0; i < MR; ++i)
#pragma unroll
        for (int t = 0; t < NT; ++t) red[wave][i * NT + t][lane] = acc[i][t];
    __syncthreads();
    // wave w finishes tiles w, w + 4, ...; lane holds D[4 kq + e][r16] of
    // activation tile i, weight group t
    for (int q = wave; q < MR * NT; q += 4) {
        const int i = q / NT, t = q - i * NT;
        f32x4 v = red[0][q][lane];
#pragma unroll
        for (int w = 1; w < 4; ++w) v += red[w][q][lane];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int m = 16 * i + 4 * kq + e;
            const float val = v[e];
            if (SPLIT) {
                if (ok[t] && m < M) p.partial[(static_cast<size_t>(blockIdx.y) * M + m) * p.Nw + n[t]] = val;
            } else if (EPI == EPI_SWIGLU) {
                const float up = __shfl(val, (lane & ~15) | ((r16 + 8) & 15), 64);
                if (r16 < 8 && ok[t] && m < M)
                    static_cast<uint16_t*>(p.act)[static_cast<size_t>(m) * p.ld_act + n[t]] =
                        f32_to_bf16(swiglu_bf16(val, up));
            } else if (ok[t] && m < M) {
                if (EPI == EPI_F32) p.out_f32[static_cast<size_t>(m) * p.ldo + n[t]] = val;
                else p.resid[static_cast<size_t>(m) * p.ldr + n[t]] += val;
            }
        }
    }
}

hipError_t launch_gemv_wide(const GemmArgs& a, const GemmPlan& p, hipStream_t s) {
    if (a.M > 64 || a.K % 64 != 0 || p.ksplit <= 0 || p.ksplit % 64 != 0 || ceil_div(a.K, p.ksplit) != p.splits ||
        p.splits > kMaxSplits)
        return hipErrorInvalidValue;
    const int groups = a.epi == EPI_SWIGLU ? ceil_div(a.F, 32) : ceil_div(a.Nw, 64);
    const int kw = ceil_div(ceil_div(p.ksplit, 4), 64) * 64;
    dim3 grid(groups, p.splits), block(256);
#define RL_GW(MR)                                                                                              \
    do {                                                                                                       \
        if (p.splits > 1) {                                                                                    \
            if (a.epi == EPI_SWIGLU)                                                                           \
                hipLaunchKernelGGL((gemv_wide_kernel<MR, EPI_SWIGLU, true>), grid, block, 0, s, a, p.ksplit, kw); \
            else hipLaunchKernelGGL((gemv_wide_kernel<MR, EPI_F32, true>), grid, block, 0, s, a, p.ksplit, kw);   \
        } else if (a.epi == EPI_F32) {                                                                         \
            hipLaunchKernelGGL((gemv_wide_kernel<MR, EPI_F32, false>), grid, block, 0, s, a, p.ksplit, kw);      \
        } else if (a.epi == EPI_RESID) {                                                                       \
            hipLaunchKernelGGL((gemv_wide_kernel<MR, EPI_RESID, false>), grid, block, 0, s, a, p.ksplit, kw);    \
        } else {                                                                                               \
            hipLaunchKernelGGL((gemv_wide_kernel<MR, EPI_SWIGLU, false>), grid, block, 0, s, a, p.ksplit, kw);   \
        }                                                                                                      \
    } while (0)
    if (a.M <= 16) RL_GW(1);
    else if (a.M <= 32) RL_GW(2);
    else RL_GW(4);
#undef RL_GW
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// split-K reduction (fixed summation order) + epilogue
// ---------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256) splitk_reduce_kernel(GemmArgs p, int splits,
        const float* __restrict__ part) {
    const int n_out = p.epi == EPI_SWIGLU ? p.F : p.Nw;
    const size_t total = static_cast<size_t>(p.M) * n_out;
    const size_t slice = static_cast<size_t>(p.M) * p.Nw;
    for (size_t idx = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x; idx < total;
         idx += static_cast<size_t>(gridDim.x) * blockDim.x) {
        const int m = static_cast<int>(idx / n_out);
        const int c = static_cast<int>(idx - static_cast<size_t>(m) * n_out);
        const float* src = part + static_cast<size_t>(m) * p.Nw + c;
        float v = 0.0f;
        for (int z = 0; z < splits; ++z) v += src[z * slice];
        if (p.epi == EPI_F32) {
            p.out_f32[static_cast<size_t>(m) * p.ldo + c] = v;
        } else if (p.epi == EPI_RESID) {
            p.resid[static_cast<size_t>(m) * p.ldr + c] += v;
        } else {
            float u = 0.0f;
            for (int z = 0; z < splits; ++z) u += src[z * slice + p.F];
            Elem<T>::store(static_cast<T*>(p.act), static_cast<size_t>(m) * p.ld_act + c, swiglu<T>(v, u));
        }
    }
}

// Four consecutive columns per thread (n_out, Nw and the output strides
// multiples of 4): 16-byte loads of every slice, issued before the in-order sum.
template <typename T>
__global__ void __launch_bounds__(256) splitk_reduce4_kernel(GemmArgs p, int splits,
        const float* __restrict__ part) {
    const int n_out = p.epi == EPI_SWIGLU ? p.F : p.Nw;
    const size_t total4 = static_cast<size_t>(p.M) * n_out / 4;
    const size_t slice = static_cast<size_t>(p.M) * p.Nw;
    for (size_t i4 = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x; i4 < total4;
         i4 += static_cast<size_t>(gridDim.x) * blockDim.x) {
        const size_t idx = 4 * i4;
        const int m = static_cast<int>(idx / n_out);
        const int c = static_cast<int>(idx - static_cast<size_t>(m) * n_out);
        const float* src = part + static_cast<size_t>(m) * p.Nw + c;
        auto sum = [&](const float* b) {
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
            int z = 0;
            for (; z + 4 <= splits; z += 4) {
                const f32x4 a0 = *reinterpret_cast<const f32x4*>(b + (z + 0) * slice);
                const f32x4 a1 = *reinterpret_cast<const f32x4*>(b + (z + 1) * slice);
                const f32x4 a2 = *reinterpret_cast<const f32x4*>(b + (z + 2) * slice);
                const f32x4 a3 = *reinterpret_cast<const f32x4*>(b + (z + 3) * slice);
                acc += a0; acc += a1; acc += a2; acc += a3;
            }
            for (; z < splits; ++z) acc += *reinterpret_cast<const f32x4*>(b + z * slice);
            return acc;
        };
        const f32x4 v = sum(src);
        if (p.epi == EPI_F32) {
            *reinterpret_cast<f32x4*>(p.out_f32 + static_cast<size_t>(m) * p.ldo + c) = v;
        } else if (p.epi == EPI_RESID) {
            f32x4* r = reinterpret_cast<f32x4*>(p.resid + static_cast<size_t>(m) * p.ldr + c);
            *r = *r + v;
        } else {
            const f32x4 u = sum(src + p.F);
            T* act = static_cast<T*>(p.act) + static_cast<size_t>(m) * p.ld_act + c;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                Elem<T>::store(act, e, swiglu<T>(v[e], u[e]));
            }
        }
    }
}

hipError_t launch_splitk_reduce(int dt, const GemmArgs& a, int splits, const float* partial,
                                hipStream_t s) {
    const int n_out = a.epi == EPI_SWIGLU ? a.F : a.Nw;
    const size_t total = static_cast<size_t>(a.M) * n_out;
    if (total == 0) return hipSuccess;
    const int ld = a.epi == EPI_F32 ? a.ldo : a.epi == EPI_RESID ? a.ldr : a.ld_act;
    const bool vec = n_out % 4 == 0 && a.Nw % 4 == 0 && ld % 4 == 0;
    size_t blocks = ((vec ? total / 4 : total) + 255) / 256;
    if (blocks > 16384) blocks = 16384;
    const dim3 grid(static_cast<unsigned>(blocks)), block(256);
    if (vec) {
        if (dt == DT_BF16) hipLaunchKernelGGL(splitk_reduce4_kernel<uint16_t>, grid, block, 0, s, a, splits, partial);
        else hipLaunchKernelGGL(splitk_reduce4_kernel<float>, grid, block, 0, s, a, splits, partial);
    } else {
        if (dt == DT_BF16) hipLaunchKernelGGL(splitk_reduce_kernel<uint16_t>, grid, block, 0, s, a, splits, partial);
        else hipLaunchKernelGGL(splitk_reduce_kernel<float>, grid, block, 0, s, a, splits, partial);
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Matrix-core rate probe: every wave runs `iters` rounds of eight independent
// 32x32x16 bf16 MFMAs (all operands 1.0, so each accumulator element gains
// 16 per MFMA), then lane 0 writes its first accumulator element summed over
// the eight chains (= 128 * iters).  No memory traffic in the loop.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256) mfma_probe_kernel(int iters, float* __restrict__ out) {
    const u32x4 ones = {0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u};   // bf16 1.0 pairs
    const bf16x8 a = as_bf16x8(ones);
    f32x16 acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[j][e] = 0.f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[j] = mfma32x32x16(a, a, acc[j]);
    }
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) s += acc[j][0];
    if ((threadIdx.x & 63) == 0) out[blockIdx.x * 4 + (threadIdx.x >> 6)] = s;
}

hipError_t launch_mfma_probe(int n_blocks, int iters, float* out, hipStream_t s) {
    if (n_blocks <= 0) return hipSuccess;
    hipLaunchKernelGGL(mfma_probe_kernel, dim3(static_cast<unsigned>(n_blocks)), dim3(256), 0, s, iters, out);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// fp32 VALU kernel: out_f32[m][n] = sum_k A[m][k] W[n][k]
// 32 x 64 output tile, 2 x 4 per thread, k tiles of 32 through LDS.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256) gemm_f32_kernel(const float* __restrict__ A, int lda,
        const float* __restrict__ W, int ldw, int M, int N, int K, float* __restrict__ out, int ldo) {
    __shared__ float As[32][33];
    __shared__ float Ws[32][65];
    const int tid = threadIdx.x;
    const int tx = tid & 15, ty = tid >> 4;
    const int m0 = blockIdx.y * 32, n0 = blockIdx.x * 64;
    float acc[2][4] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
    for (int k0 = 0; k0 < K; k0 += 32) {
        for (int e = tid; e < 32 * 32; e += 256) {
            const int r = e >> 5, k = e & 31;
            const int m = m0 + r, kk = k0 + k;
            As[k][r] = (m < M && kk < K) ? A[static_cast<size_t>(m) * lda + kk] : 0.0f;
        }
        for (int e = tid; e < 64 * 32; e += 256) {
            const int r = e >> 5, k = e & 31;
            const int n = n0 + r, kk = k0 + k;
            Ws[k][r] = (n < N && kk < K) ? W[static_cast<size_t>(n) * ldw + kk] : 0.0f;
        }
        __syncthreads();
#pragma unroll 8
        for (int k = 0; k < 32; ++k) {
            const float a0 = As[k][ty * 2], a1 = As[k][ty * 2 + 1];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float w = Ws[k][tx * 4 + j];
                acc[0][j] = fmaf(a0, w, acc[0][j]);
                acc[1][j] = fmaf(a1, w, acc[1][j]);
            }
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int m = m0 + ty * 2 + i;
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int n = n0 + tx * 4 + j;
            if (n < N) out[static_cast<size_t>(m) * ldo + n] = acc[i][j];
        }
    }
}

hipError_t launch_gemm_f32(const GemmArgs& a, hipStream_t s) {
    if (a.M <= 0) return hipSuccess;
    dim3 grid(ceil_div(a.Nw, 64), ceil_div(a.M, 32));
    hipLaunchKernelGGL(gemm_f32_kernel, grid, dim3(256), 0, s, static_cast<const float*>(a.A), a.lda,
                       static_cast<const float*>(a.W), a.ldw, a.M, a.Nw, a.K, a.out_f32, a.ldo);
    return hipGetLastError();
}

}  // namespace rl
