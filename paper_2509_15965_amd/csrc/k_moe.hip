// k_moe.hip -- mixture-of-experts MLP (the Qwen3-30B-A3B policy of the
// paper's Sec. 5.1.1): top-k routing of the router logits, the (row, choice)
// pairs grouped by expert, and the grouped expert projections.
//
// A step's n rows make n * k pairs p = row * k + j (j-th choice of row).
// After grouping, pairs[off[e] .. off[e+1]) lists the pairs that chose
// expert e; the gate|up projection writes each pair's SwiGLU row at its
// position in that list, and the down projection writes w_p times its
// output into plane j of row `row` ([k][n][H] fp32), which the residual +
// RMSNorm kernel sums in plane order (as it sums split-K slices).  A pair's
// outputs do not depend on where it sits in the list, so the order inside an
// expert's range (set by LDS atomics) does not change any result.
#include "rl_device.h"
#include "rl_internal.h"

namespace rl {

namespace {

constexpr int kMoeMaxPerLane = kMoeMaxExperts / 64;

// One wave per row: the k largest logits (equal values: the lower expert
// first; NaN ranks below every number, so k valid experts are always
// chosen), then w_j = softmax of the chosen logits.
__global__ void __launch_bounds__(256) moe_topk_kernel(const float* __restrict__ logits, int n, int E, int k,
                                                       int32_t* __restrict__ ids, float* __restrict__ w) {
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= n) return;
    const float* r = logits + static_cast<size_t>(row) * E;
    float v[kMoeMaxPerLane];
#pragma unroll
    for (int i = 0; i < kMoeMaxPerLane; ++i) {
        const int e = lane + 64 * i;
        const float x = e < E ? r[e] : -INFINITY;
        v[i] = x != x ? -INFINITY : x;
    }
    uint32_t taken = 0;
    float v0 = 0.0f, mine_v = -INFINITY;
    int mine_i = 0;
    for (int j = 0; j < k; ++j) {
        float bv = -INFINITY;
        int bi = 0x7fffffff;
#pragma unroll
        for (int i = 0; i < kMoeMaxPerLane; ++i) {
            const int e = lane + 64 * i;
            if (e < E && !((taken >> i) & 1u) && (v[i] > bv || (v[i] == bv && e < bi))) {
                bv = v[i];
                bi = e;
            }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            const float ov = __shfl_xor(bv, o, 64);
            const int oi = __shfl_xor(bi, o, 64);
            if (ov > bv || (ov == bv && oi < bi)) {
                bv = ov;
                bi = oi;
            }
        }
        if (lane == (bi & 63)) taken |= 1u << (bi >> 6);
        if (j == 0) v0 = bv;
        if (lane == j) {
            mine_v = bv;
            mine_i = bi;
        }
    }
    float ex = lane < k ? expf(mine_v - v0) : 0.0f;
    float sum = ex;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o, 64);
    if (lane < k) {
        ids[static_cast<size_t>(row) * k + lane] = mine_i;
        w[static_cast<size_t>(row) * k + lane] = ex / sum;
    }
}

// Pairs grouped by expert (one workgroup): counts, an exclusive scan, then
// each pair's slot in its expert's range.
__global__ void __launch_bounds__(1024) moe_group_kernel(const int32_t* __restrict__ ids, int npairs, int E,
                                                         int32_t* __restrict__ off, int32_t* __restrict__ pairs) {
    __shared__ int32_t cnt[kMoeMaxExperts];
    __shared__ int32_t scan[kMoeMaxExperts];
    const int t = threadIdx.x;
    cnt[t] = 0;
    __syncthreads();
    for (int p = t; p < npairs; p += 1024) {
        const int e = min(max(ids[p], 0), E - 1);
        atomicAdd(&cnt[e], 1);
    }
    __syncthreads();
    // inclusive scan of the counts (Hillis-Steele over the 1024 threads)
    scan[t] = cnt[t];
    __syncthreads();
    for (int d = 1; d < kMoeMaxExperts; d <<= 1) {
        const int add = t >= d ? scan[t - d] : 0;
        __syncthreads();
        scan[t] += add;
        __syncthreads();
    }
    const int base = scan[t] - cnt[t];   // exclusive
    if (t < E) off[t] = base;
    if (t == E - 1) off[E] = scan[t];
    __syncthreads();
    cnt[t] = base;   // next free slot of expert t
    __syncthreads();
    for (int p = t; p < npairs; p += 1024) {
        const int e = min(max(ids[p], 0), E - 1);
        pairs[atomicAdd(&cnt[e], 1)] = p;
    }
}

// Grouped expert projection: workgroup (e, g) owns 16 * NT weight rows of
// expert e (SwiGLU: NT groups of 8 gate rows and the matching 8 up rows) and
// the whole K, and runs every pair of e through them, 16 * MR pairs at a
// time, so each pair row it gathers serves NT row groups.  Wave w takes the
// w-th quarter of K; the four partial tiles are summed through LDS in wave
// order.
template <int MR, int NT, int EPI>
__global__ void __launch_bounds__(256) moe_gemv_kernel(MoeArgs a, int kw) {
    constexpr int U = 2;   // 64-wide k blocks per batch of loads
    __shared__ f32x4 red[4][MR * NT][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r16 = lane & 15, kq = lane >> 4;
    const int e = blockIdx.x / a.groups, g = blockIdx.x - e * a.groups;
    const int p0 = min(max(a.off[e], 0), a.npairs), p1 = min(max(a.off[e + 1], p0), a.npairs);
    if (p0 == p1) return;

    int n[NT];
    bool ok[NT];
    const uint16_t* wp[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        if (EPI == EPI_SWIGLU) {
            const int c = (g * NT + t) * 8 + (r16 & 7);
            ok[t] = c < a.F;
            n[t] = r16 < 8 ? c : a.F + c;
        } else {
            n[t] = (g * NT + t) * 16 + r16;
            ok[t] = n[t] < a.Nw;
        }
        wp[t] = a.W + static_cast<size_t>(e) * a.w_expert + static_cast<size_t>(ok[t] ? n[t] : 0) * a.ldw + 8 * kq;
    }
    const int kb = wave * kw;
    const int ke = min(a.K, kb + kw);
    const u32x4 zero = {0u, 0u, 0u, 0u};

    for (int c0 = p0; c0 < p1; c0 += 16 * MR) {
        const uint16_t* ap[MR];
        bool aok[MR];
#pragma unroll
        for (int i = 0; i < MR; ++i) {
            const int pos = c0 + 16 * i + r16;
            aok[i] = pos < p1;
            // gate|up reads the pair's token row; down reads the pair's SwiGLU row
            const int arow = !aok[i] ? 0 : EPI == EPI_SWIGLU ? a.pairs[pos] / a.k : pos;
            ap[i] = a.A + static_cast<size_t>(arow) * a.lda + 8 * kq;
        }
        f32x4 acc[MR][NT];
#pragma unroll
        for (int i = 0; i < MR; ++i)
#pragma unroll
            for (int t = 0; t < NT; ++t) acc[i][t] = f32x4{0.f, 0.f, 0.f, 0.f};
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
        // wave w finishes tiles w, w + 4, ...: the four waves' partials summed in
        // order; lane holds D[4 kq + e4][r16] of pair tile i, row group t
        for (int q = wave; q < MR * NT; q += 4) {
            const int i = q / NT, t = q - i * NT;
            f32x4 v = red[0][q][lane];
#pragma unroll
            for (int w = 1; w < 4; ++w) v += red[w][q][lane];
#pragma unroll
            for (int e4 = 0; e4 < 4; ++e4) {
                const int pos = c0 + 16 * i + 4 * kq + e4;
                const float val = v[e4];
                if (EPI == EPI_SWIGLU) {
                    const float up = __shfl(val, (lane & ~15) | ((r16 + 8) & 15), 64);
                    if (r16 < 8 && ok[t] && pos < p1)
                        a.act[static_cast<size_t>(pos) * a.ld_act + n[t]] = f32_to_bf16(swiglu_bf16(val, up));
                } else if (ok[t] && pos < p1) {
                    const int p = a.pairs[pos];
                    const int row = p / a.k, j = p - row * a.k;
                    a.plane[(static_cast<size_t>(j) * a.n_rows + row) * a.Nw + n[t]] = a.pw[p] * val;
                }
            }
        }
        __syncthreads();   // red is reused by the next chunk
    }
}

}  // namespace

hipError_t launch_moe_route(const float* logits, int n, int E, int k, int32_t* ids, float* w, int32_t* off,
                            int32_t* pairs, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    if (E < 1 || E > kMoeMaxExperts || k < 1 || k > E || k > kMoeMaxTopK) return hipErrorInvalidValue;
    hipLaunchKernelGGL(moe_topk_kernel, dim3((n + 3) / 4), dim3(256), 0, s, logits, n, E, k, ids, w);
    hipLaunchKernelGGL(moe_group_kernel, dim3(1), dim3(1024), 0, s, ids, n * k, E, off, pairs);
    return hipGetLastError();
}

hipError_t launch_moe_gemv(const MoeArgs& a, int epi, hipStream_t s) {
    if (a.npairs <= 0) return hipSuccess;
    if (a.groups != (epi == EPI_SWIGLU ? (a.F + kMoeRowsPerGroup / 2 - 1) / (kMoeRowsPerGroup / 2)
                                       : (a.Nw + kMoeRowsPerGroup - 1) / kMoeRowsPerGroup))
        return hipErrorInvalidValue;
    const int kw = ((a.K + 3) / 4 + 63) / 64 * 64;
    dim3 grid(a.E * a.groups), block(256);
    constexpr int NT = kMoeRowsPerGroup / 16;
    if (epi == EPI_SWIGLU) hipLaunchKernelGGL((moe_gemv_kernel<4, NT, EPI_SWIGLU>), grid, block, 0, s, a, kw);
    else hipLaunchKernelGGL((moe_gemv_kernel<4, NT, EPI_RESID>), grid, block, 0, s, a, kw);
    return hipGetLastError();
}

}  // namespace rl
