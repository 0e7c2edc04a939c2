// k_sample.hip -- temperature log-softmax, Gumbel-max sampling and the
// per-token log-probability, one workgroup per (output row, vocabulary
// chunk); the exact noise is evaluated only where an entry can still win.
//
// Noise: Philox4x32-10 (Salmon et al., SC'11) keyed by the 64-bit seed with
// counter (v / 4, position of the new token, uid lo, uid hi); word v % 4 of
// the block is the noise word x_v of vocabulary entry v.  u = (x + 1/2) 2^-32,
// g = fl32(-log(-log u)) evaluated in fp64.  The sample is the arg-max of
// fl32(z_v / T + g_v) with ties to the lowest index; the log-probability is
// z_y / T - LSE(z / T).  T == 0: arg-max of z, log-probability at T = 1.
// The arg-max (ties to the lowest index) and the merge order are fixed, so
// the result does not depend on how the vocabulary is split.
#include "rl_device.h"
#include "rl_internal.h"

#include <mutex>
#include <vector>

namespace rl {

__device__ __forceinline__ void philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1) {
    constexpr uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
    constexpr uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r > 0) { k0 += W0; k1 += W1; }
        const uint64_t p0 = static_cast<uint64_t>(M0) * c[0], p1 = static_cast<uint64_t>(M1) * c[2];
        const uint32_t hi0 = static_cast<uint32_t>(p0 >> 32), lo0 = static_cast<uint32_t>(p0);
        const uint32_t hi1 = static_cast<uint32_t>(p1 >> 32), lo1 = static_cast<uint32_t>(p1);
        const uint32_t n0 = hi1 ^ c[1] ^ k0;
        const uint32_t n2 = hi0 ^ c[3] ^ k1;
        c[0] = n0; c[1] = lo1; c[2] = n2; c[3] = lo0;
    }
}

__device__ __forceinline__ float gumbel_of_word(uint32_t x) {
    const double u = (static_cast<double>(x) + 0.5) * 2.3283064365386963e-10;
    return static_cast<float>(-log(-log(u)));
}

// Upper bounds of g(x) = gumbel_of_word(x).  g grows with x: g < 5.56 for
// x < 0xFF000000 (u < 1 - 2^-8, g(0xFEFFFFFF) = 5.5433) and g <= 22.874 for
// every x (u = 1 - 2^-33).  Below 0xFF000000 a tighter bound comes from fp32
// hardware logarithms: rounding u to fp32 (relative error <= 2^-23) moves
// L = -ln u (>= 3.9e-3) by a relative 3.1e-5 at most, the two logarithms and
// the products add ~1e-6 each, so the fp32 value is within 1e-4 of -ln L;
// 0.01 is added on top.
constexpr uint32_t kGumbelLowWords = 0xFF000000u;
constexpr float kGumbelLowMax = 5.56f, kGumbelMax = 22.9f;
__device__ __forceinline__ float gumbel_upper_low(uint32_t x) {
    const float u = (static_cast<float>(x) + 0.5f) * 2.3283064365386963e-10f;
    const float L = -__log2f(u) * 0.69314718f;
    return -__log2f(L) * 0.69314718f + 0.01f;
}

struct Best { float s; int v; };
__device__ __forceinline__ Best better(Best a, Best b) {
    if (b.s > a.s || (b.s == a.s && b.v < a.v)) return b;
    return a;
}
struct Lse { float m, s; };
__device__ __forceinline__ Lse lse_merge(Lse a, Lse b) {
    if (a.m == -INFINITY) return b;
    if (b.m == -INFINITY) return a;
    const float m = fmaxf(a.m, b.m);
    return Lse{m, a.s * expf(a.m - m) + b.s * expf(b.m - m)};
}

// The row's token (the arg-max) and the log-probability of the token, or of
// `forced` when it is a vocabulary index.  A NaN score never wins a
// comparison, so a row whose every score is NaN ranks no entry and keeps
// the initial index: its token is -1 and its log-probability NaN (z is never
// read at an index outside [0, V)).
__device__ __forceinline__ void sample_finish(Best b, Lse a, const float* z, int V, int forced, float T, int o,
                                              int32_t* out_tok, float* out_logp) {
    const float lse = a.m + logf(a.s);
    const bool ranked = b.v >= 0 && b.v < V;
    const int r = (forced >= 0 && forced < V) ? forced : ranked ? b.v : -1;
    out_tok[o] = ranked ? b.v : -1;
    if (r < 0) {
        out_logp[o] = __builtin_nanf("");
        return;
    }
    const float zr = T == 0.0f ? z[r] : z[r] / T;
    out_logp[o] = zr - lse;
}

// One workgroup per (row, vocabulary chunk).  With several chunks per row,
// each writes its (best score, index, max, sum-exp) and sample_merge_kernel
// merges them in chunk order (a kernel boundary instead of device-scope
// fences: on this multi-XCD part a fence writes back the whole L2).
__global__ void __launch_bounds__(256) sample_kernel(const float* __restrict__ logits, int ld,
        int V, const int32_t* __restrict__ logit_row, const uint64_t* __restrict__ uid,
        const int32_t* __restrict__ pos_new, const int32_t* __restrict__ forced, uint32_t seed_lo,
        uint32_t seed_hi, float T, int chunk, SamplePart* __restrict__ parts,
        int32_t* __restrict__ out_tok, float* __restrict__ out_logp) {
    __shared__ Best sb[4];
    __shared__ Lse sl[4];
    const int o = blockIdx.x, c = blockIdx.y, nchunks = gridDim.y;
    const int row = logit_row ? logit_row[o] : o;
    const float* z = logits + static_cast<size_t>(row) * ld;
    const uint64_t u64 = uid[o];
    const uint32_t pos = static_cast<uint32_t>(pos_new[o]);
    const bool greedy = T == 0.0f;
    const bool unit_t = T == 1.0f;   // z / 1 == z exactly: no division
    const int vbeg = c * chunk, vend = min(V, vbeg + chunk);

    // The exact fp64 noise is evaluated only where the score could still
    // reach the wave's best so far: with an upper bound b >= g(x) and rounding
    // monotonic, fl32(z/T + b) < thr implies fl32(z/T + g) < thr, and thr
    // is the score of an entry already seen, so the skipped entry can neither
    // win nor tie.  The sample is therefore the same as scoring every entry.
    Best best{-INFINITY, 0x7FFFFFFF};
    Lse acc{-INFINITY, 0.0f};
    float thr = -INFINITY;
    // every lane runs the same number of iterations (the wave-wide threshold
    // reads every lane); lanes past the chunk's end score nothing
    // (the next iteration's logits are loaded before this one's math)
    auto load4 = [&](int bb) {
        const int v4 = bb + static_cast<int>(threadIdx.x);
        return 4 * v4 < vend ? *reinterpret_cast<const float4*>(z + 4 * static_cast<size_t>(v4))
                             : make_float4(0.f, 0.f, 0.f, 0.f);
    };
    float4 znext = load4(vbeg / 4);
    for (int b4 = vbeg / 4; 4 * b4 < vend; b4 += blockDim.x) {
        const int v4 = b4 + threadIdx.x;
        const float4 zz = znext;
        if (4 * (b4 + static_cast<int>(blockDim.x)) < vend) znext = load4(b4 + blockDim.x);
        const float zv[4] = {zz.x, zz.y, zz.z, zz.w};
        uint32_t cw[4] = {static_cast<uint32_t>(v4), pos, static_cast<uint32_t>(u64),
                          static_cast<uint32_t>(u64 >> 32)};
        if (!greedy) philox4x32_10(cw, seed_lo, seed_hi);
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const int v = 4 * v4 + w;
            if (v >= vend) break;
            const float zt = greedy || unit_t ? zv[w] : zv[w] / T;
            if (greedy) {
                best = better(best, Best{zt, v});
            } else {
                const uint32_t x = cw[w];
                const bool cand = x >= kGumbelLowWords
                                      ? !(zt + kGumbelMax < thr)
                                      : !(zt + kGumbelLowMax < thr) && !(zt + gumbel_upper_low(x) < thr);
                if (cand) best = better(best, Best{zt + gumbel_of_word(x), v});
            }
            if (zt > acc.m) {
                acc.s = acc.s * __expf(acc.m - zt) + 1.0f;
                acc.m = zt;
            } else {
                acc.s += __expf(zt - acc.m);
            }
        }
        float t = best.s;
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) t = fmaxf(t, __shfl_xor(t, off, 64));
        thr = t;
    }
    for (int off = 32; off > 0; off >>= 1) {
        Best ob{__shfl_xor(best.s, off, 64), __shfl_xor(best.v, off, 64)};
        best = better(best, ob);
        Lse ol{__shfl_xor(acc.m, off, 64), __shfl_xor(acc.s, off, 64)};
        acc = lse_merge(acc, ol);
    }
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) { sb[wave] = best; sl[wave] = acc; }
    __syncthreads();
    if (threadIdx.x != 0) return;
    Best b = sb[0];
    Lse a = sl[0];
    for (int w = 1; w < 4; ++w) { b = better(b, sb[w]); a = lse_merge(a, sl[w]); }
    if (nchunks > 1) {   // merged by sample_merge_kernel
        parts[static_cast<size_t>(o) * nchunks + c] = SamplePart{b.s, b.v, a.m, a.s};
        return;
    }
    sample_finish(b, a, z, V, forced ? forced[o] : -1, T, o, out_tok, out_logp);
}

// One 64-lane workgroup per row: lane k loads chunk k's partial (all in one
// memory round trip), then lane 0 merges them in chunk order.
__global__ void __launch_bounds__(64) sample_merge_kernel(const SamplePart* __restrict__ parts, int nchunks,
        const float* __restrict__ logits, int ld, int V, const int32_t* __restrict__ logit_row,
        const int32_t* __restrict__ forced, float T, int32_t* __restrict__ out_tok, float* __restrict__ out_logp) {
    __shared__ SamplePart sp[kSampleMaxChunks];
    const int o = blockIdx.x;
    const SamplePart* pr = parts + static_cast<size_t>(o) * nchunks;
    for (int k = threadIdx.x; k < nchunks; k += blockDim.x) sp[k] = pr[k];
    __syncthreads();
    if (threadIdx.x != 0) return;
    Best b{sp[0].best_s, sp[0].best_v};
    Lse a{sp[0].m, sp[0].s};
    for (int k = 1; k < nchunks; ++k) {
        b = better(b, Best{sp[k].best_s, sp[k].best_v});
        a = lse_merge(a, Lse{sp[k].m, sp[k].s});
    }
    const int row = logit_row ? logit_row[o] : o;
    sample_finish(b, a, logits + static_cast<size_t>(row) * ld, V, forced ? forced[o] : -1, T, o, out_tok, out_logp);
}

// Check of the noise bounds the sampler relies on, over the words
// [lo, lo + count): for x < kGumbelLowWords, gumbel_upper_low(x) >= g(x) and
// kGumbelLowMax >= g(x); above, kGumbelMax >= g(x).  Each workgroup writes its
// count of violations and its smallest margin gumbel_upper_low(x) - g(x).
__global__ void __launch_bounds__(256) gumbel_bound_probe_kernel(uint32_t lo, uint64_t count,
                                                                 uint32_t* __restrict__ viol,
                                                                 float* __restrict__ min_margin) {
    __shared__ uint32_t sv[4];
    __shared__ float sm[4];
    uint32_t bad = 0;
    float mm = INFINITY;
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * blockDim.x;
    for (uint64_t i = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < count; i += stride) {
        const uint32_t x = lo + static_cast<uint32_t>(i);
        const float g = gumbel_of_word(x);
        if (x < kGumbelLowWords) {
            const float b = gumbel_upper_low(x);
            bad += !(b >= g);
            bad += !(kGumbelLowMax >= g);
            mm = fminf(mm, b - g);
        } else {
            bad += !(kGumbelMax >= g);
        }
    }
    for (int off = 32; off > 0; off >>= 1) {
        bad += __shfl_xor(bad, off, 64);
        mm = fminf(mm, __shfl_xor(mm, off, 64));
    }
    if ((threadIdx.x & 63) == 0) { sv[threadIdx.x >> 6] = bad; sm[threadIdx.x >> 6] = mm; }
    __syncthreads();
    if (threadIdx.x == 0) {
        viol[blockIdx.x] = sv[0] + sv[1] + sv[2] + sv[3];
        min_margin[blockIdx.x] = fminf(fminf(sm[0], sm[1]), fminf(sm[2], sm[3]));
    }
}

hipError_t launch_gumbel_bound_probe(uint32_t lo, uint64_t count, int n_blocks, uint32_t* viol,
                                     float* min_margin, hipStream_t s) {
    hipLaunchKernelGGL(gumbel_bound_probe_kernel, dim3(n_blocks), dim3(256), 0, s, lo, count, viol, min_margin);
    return hipGetLastError();
}

// Vocabulary split of a sampling launch: about 2048 workgroups in all, chunks
// of whole 1024-entry blocks, at most kSampleMaxChunks per row.
static void sample_split(int n, int V, int* nchunks_out, int* chunk_out) {
    int nchunks = (2048 + n - 1) / n;
    nchunks = nchunks < 1 ? 1 : nchunks > kSampleMaxChunks ? kSampleMaxChunks : nchunks;
    int chunk = (V + nchunks - 1) / nchunks;
    chunk = (chunk + 1023) / 1024 * 1024;
    *nchunks_out = (V + chunk - 1) / chunk;
    *chunk_out = chunk;
}

size_t sample_parts_needed(int n, int V) {
    if (n <= 0) return 0;
    int nchunks, chunk;
    sample_split(n, V, &nchunks, &chunk);
    return nchunks > 1 ? static_cast<size_t>(n) * nchunks : 0;
}

hipError_t launch_sample(const float* logits, int ld, int n, int V, const int32_t* logit_row,
                         const uint64_t* uid, const int32_t* pos_new, const int32_t* forced,
                         uint64_t seed, float T, SamplePart* parts,
                         int32_t* out_tok, float* out_logp, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    int nchunks, chunk;
    sample_split(n, V, &nchunks, &chunk);
    hipLaunchKernelGGL(sample_kernel, dim3(n, nchunks), dim3(256), 0, s, logits, ld, V, logit_row, uid,
                       pos_new, forced, static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32),
                       T, chunk, parts, out_tok, out_logp);
    if (nchunks > 1)
        hipLaunchKernelGGL(sample_merge_kernel, dim3(n), dim3(64), 0, s, parts, nchunks, logits, ld, V, logit_row,
                           forced, T, out_tok, out_logp);
    return hipGetLastError();
}

// Inference-stage log-probabilities of given tokens, one workgroup per logits
// row: the row's LSE of fl32(z / T) (online max / sum-exp per lane, merged in
// a fixed lane and wave order), then every item of the row.  No noise.
__global__ void __launch_bounds__(256) logprob_kernel(const float* __restrict__ logits, int ld, int V,
        const int32_t* __restrict__ row_items, const int32_t* __restrict__ item_idx,
        const int32_t* __restrict__ targets, float T, float* __restrict__ out) {
    __shared__ Lse sl[4];
    const int r = blockIdx.x;
    const float* z = logits + static_cast<size_t>(r) * ld;
    Lse acc{-INFINITY, 0.0f};
    for (int v4 = threadIdx.x; 4 * v4 < V; v4 += blockDim.x) {
        const float4 zz = *reinterpret_cast<const float4*>(z + 4 * static_cast<size_t>(v4));
        const float zv[4] = {zz.x / T, zz.y / T, zz.z / T, zz.w / T};
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const float zt = zv[w];
            if (zt > acc.m) {
                acc.s = acc.s * expf(acc.m - zt) + 1.0f;
                acc.m = zt;
            } else {
                acc.s += expf(zt - acc.m);
            }
        }
    }
    for (int off = 32; off > 0; off >>= 1) {
        Lse o{__shfl_xor(acc.m, off, 64), __shfl_xor(acc.s, off, 64)};
        acc = lse_merge(acc, o);
    }
    if ((threadIdx.x & 63) == 0) sl[threadIdx.x >> 6] = acc;
    __syncthreads();
    Lse a = sl[0];
    for (int w = 1; w < 4; ++w) a = lse_merge(a, sl[w]);
    const float lse = a.m + logf(a.s);
    for (int k = row_items[r] + threadIdx.x; k < row_items[r + 1]; k += blockDim.x) {
        const int idx = item_idx[k];
        const int y = targets[idx];
        out[idx] = (y >= 0 && y < V) ? z[y] / T - lse : __builtin_nanf("");
    }
}

hipError_t launch_logprob(const float* logits, int ld, int n_rows, int V, const int32_t* row_items,
                          const int32_t* item_idx, const int32_t* targets, float T, float* out,
                          hipStream_t s) {
    if (n_rows <= 0) return hipSuccess;
    hipLaunchKernelGGL(logprob_kernel, dim3(n_rows), dim3(256), 0, s, logits, ld, V, row_items, item_idx,
                       targets, T, out);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Allocation-free sampling: the chunk partials live in a file-scope device
// array instead of a caller's workspace.  Each device the library runs on
// holds its own copy until the process ends; host code reaches it only
// through the address hipGetSymbolAddress returns on that device.
// ---------------------------------------------------------------------------
static __device__ __align__(256) SamplePart scratch[kStaticSampleParts];

hipError_t static_sample_parts(SamplePart** out) {
    static std::mutex mu;
    static std::vector<SamplePart*> addr;   // per device ordinal
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lock(mu);
    if (static_cast<size_t>(dev) >= addr.size()) addr.resize(static_cast<size_t>(dev) + 1, nullptr);
    if (!addr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[dev] = static_cast<SamplePart*>(p);
    }
    *out = addr[dev];
    return hipSuccess;
}

}  // namespace rl
