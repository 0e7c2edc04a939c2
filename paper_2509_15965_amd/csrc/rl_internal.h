// rl_internal.h -- declarations shared by the HIP kernels and the host engine
// of the rollout decode library (not part of the public C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace rl {

// Element encodings of the model dtype.
enum DType { DT_F32 = 0, DT_BF16 = 1 };

// Where the K/V of (slot, position) lives.  The K slab is blocks of
// [page][d] and the V slab blocks of [page/8][d][8], one per (layer, page,
// kv-head) in that order, `stride` elements apart (>= page * d).
// table == nullptr: slot s is page s and holds all `page` (= the slot
// capacity) positions.  Otherwise position p of slot s is in page
// table[s * maxp + p / page] at p % page (page a multiple of 32, so a
// 32-position step never straddles pages).
struct KvPages {
    const int32_t* table;
    int maxp;
    int page;
    int pages;
    size_t stride;
};

// Page of (slot, pos) and the position inside it; an id outside the pool is
// clamped into it (the host never stores one; this only keeps every address
// inside the slab).
__device__ __forceinline__ int kv_clamp(const KvPages& kp, int pid) {
    return pid < 0 ? 0 : pid >= kp.pages ? kp.pages - 1 : pid;
}
// Table entry j (< maxp) of a slot, as stored.
__device__ __forceinline__ int kv_table(const KvPages& kp, int slot, int j) {
    return kp.table[static_cast<size_t>(slot) * kp.maxp + j];
}
__device__ __forceinline__ int kv_page(const KvPages& kp, int slot, int pos, int* local) {
    if (!kp.table) {
        *local = pos;
        return slot;
    }
    const int j = pos / kp.page;
    *local = pos - j * kp.page;
    return kv_clamp(kp, kv_table(kp, slot, j));
}

// Element offset of the K (or V) block of (layer, page, kv-head).
__device__ __forceinline__ size_t kv_block(const KvPages& kp, int layer, int Hkv, int pid, int head) {
    return ((static_cast<size_t>(layer) * kp.pages + pid) * Hkv + head) * kp.stride;
}

// GEMM epilogues: Y = X . W^T followed by
enum Epi {
    EPI_F32 = 0,      // store fp32 Y
    EPI_RESID = 1,    // fp32 residual += Y
    EPI_SWIGLU = 2    // act[m][c] = storage(silu(Y[m][c]) * Y[m][F + c]), c < F
};

// One split-KV attention work item: a block of nq consecutive query tokens
// of one sequence (nq * group <= 16 columns) against key positions
// [kv_lo, kv_hi) of one KV slot.  kv_lo is a multiple of 32.
struct AttnItem {
    int32_t qrow;   // workspace row of the first query token
    int32_t nq;     // query tokens in the block
    int32_t slot;   // KV slot read
    int32_t pos0;   // position of the first query token
    int32_t kv_lo;
    int32_t kv_hi;
    int32_t part;   // partial-sum index, or -1 when this item covers every key
                    // its tokens see (it then writes the final output)
    int32_t part0;  // first partial index of the block's items (they are consecutive)
    int32_t nparts; // items of the block (>= 2 when part >= 0)
    int32_t qrow_b; // >= 0: a pair item over a shared prompt chunk -- columns
                    // [G, 2G) are the single token of a second sequence,
                    // workspace row qrow_b, partial index part_b (nq = 2,
                    // no key of the chunk is masked for either); -1: none
    int32_t part_b;
    int32_t pad;    // 1 on the first item of a workgroup whose four items read
                    // the same shared prompt chunk (same slot and key range):
                    // the workgroup stages each K/V step through LDS once
};

struct GemmArgs {
    const void* A;   int lda;     // [M][K] model dtype
    const void* W;   int ldw;     // [Nw][K] model dtype (Nw = 2F for SwiGLU)
    int M, Nw, K;
    int epi;
    float* out_f32;  int ldo;     // EPI_F32
    float* resid;    int ldr;     // EPI_RESID
    void* act;       int ld_act;  // EPI_SWIGLU output, model dtype
    int F;                        // EPI_SWIGLU
    float* partial;               // [splits][M][Nw] when splits > 1
};

// Mixture of experts: one grouped expert projection (k_moe.hip).
constexpr int kMoeMaxExperts = 1024;
constexpr int kMoeMaxTopK = 16;
constexpr int kMoeRowsPerGroup = 64;   // weight rows of one expert per workgroup (SwiGLU: 32 gate + 32 up)
struct MoeArgs {
    const uint16_t* A; int lda;            // gate|up: token rows [n][K]; down: the pairs' SwiGLU rows [n*k][K]
    const uint16_t* W; size_t w_expert;    // expert e's matrix at W + e * w_expert, rows [Nw][K]
    int ldw, K, Nw, F;                     // F: SwiGLU width (gate|up only; Nw = 2F)
    int E, groups, k, n_rows, npairs;      // groups: kMoeRowsPerGroup-row weight groups per expert
    const int32_t* off;                    // [E + 1] ranges of pairs per expert
    const int32_t* pairs;                  // [n*k] pair index p = row * k + j, grouped by expert
    const float* pw;                       // [n*k] routing weight of pair p (down only)
    uint16_t* act; int ld_act;             // gate|up output: SwiGLU row of each pair position
    float* plane;                          // down output: [k][n_rows][Nw], plane j of row `row`
};

struct GemmPlan {
    int variant;   // tile kernel (index into the tile-shape table or a k*Variant id)
    int splits;
    int ksplit;    // K elements per split (multiple of 64)
    int grid_x, grid_y;
    int n_split;   // output columns [n_split, n_out) use variant2, without split-K
    int variant2;  //   (n_split == 0: one segment)
};

// Tile shapes of the bf16 MFMA GEMM: wave tile (16*MT) x (16*NT) weight rows,
// 4 waves per workgroup arranged WR x WC.
struct GemmShape { int MT, NT, WR, WC; };
constexpr int kNumGemmShapes = 3;           // direct-load shapes for M <= 64
extern const GemmShape kGemmShapes[kNumGemmShapes];
constexpr int kLdsVariant128 = 3;           // register-staged LDS 128 x 128 (K % 32 != 0)
constexpr int kLdsVariant256 = 4;           // register-staged LDS 256 x 128 (K % 32 != 0)
constexpr int kDmaVariant256x256 = 5;       // direct-to-LDS, 64-byte rows, 256 x 256, 8 waves (K % 32 == 0)
constexpr int kDmaVariant128x256 = 6;       // direct-to-LDS, 64-byte rows, 128 x 256, 8 waves (K % 32 == 0)
constexpr int kLineVariant256x256 = 7;      // direct-to-LDS, 128-byte rows, 256 x 256, 8 waves (K % 64 == 0)
constexpr int kLineVariant128x128 = 8;      // direct-to-LDS, 128-byte rows, 128 x 128, 4 waves, 2 per CU
constexpr int kLineVariant128x256 = 9;      // direct-to-LDS, 128-byte rows, 128 x 256, 8 waves
constexpr int kLineVariant128x128Deep = 10; // direct-to-LDS, 128-byte rows, 128 x 128, 4 waves, 4-stage ring
constexpr int kGemvVariant = 11;            // M <= 32: 16 weight rows x all K per 8-wave workgroup, no split-K
constexpr int kGemvWideVariant = 12;        // M <= 64: 64 weight rows x a K slice per 4-wave workgroup

constexpr int kMaxSplits = 32;
constexpr size_t kPartCapFloats = size_t(32) << 20;   // split-K partials budget

GemmPlan plan_gemm_bf16(int M, int Nw, int K, int epi, int F);
// the cost model's search space, its choice first; returns the count (<= cap)
int plan_gemm_candidates(int M, int Nw, int K, int epi, int F, GemmPlan* out, int cap);
// RL_OPT_GEMM_PLAN code of a plan (0: none)
int64_t gemm_plan_code_of(const GemmPlan& p);
constexpr int kMaxGemmCandidates = 48;
// RL_OPT_GEMM_PLAN override; false when it cannot serve this GEMM
bool plan_gemm_forced(int M, int Nw, int K, int epi, int F, int64_t code, GemmPlan* p);

// ---- launchers (enqueue only; return hipGetLastError()) -----------------
// x = embedding rows; h = first-layer attention norm of x when h != nullptr
hipError_t launch_embed(int dt, const int32_t* tok, int n, const void* table, int V,
                        const void* rows, int n_rows, int H, float* x, const void* g, float eps, void* h,
                        hipStream_t s);

hipError_t launch_rmsnorm(int dt, const float* x, const int32_t* sel, int n, int H,
                          const void* g, float eps, void* out, hipStream_t s);

// x[r] += sum of `splits` split-K slices [splits][n][H] (in order), then
// out[r] = storage(rmsnorm(x[r]) * g); one workgroup per row (H % 4 == 0, H <= 8192)
hipError_t launch_resid_norm(int dt, const float* part, int splits, float* x, int n, int H, const void* g,
                             float eps, void* out, hipStream_t s);

hipError_t launch_gemm_bf16(const GemmArgs& a, const GemmPlan& p, hipStream_t s);
hipError_t launch_gemm_bf16_lds(const GemmArgs& a, const GemmPlan& p, hipStream_t s);
hipError_t launch_gemm_f32(const GemmArgs& a, hipStream_t s);   // writes a.out_f32 [M][Nw]
hipError_t launch_splitk_reduce(int dt, const GemmArgs& a, int splits, const float* partial,
                                hipStream_t s);

// RoPE on q and k of fp32 q|k|v rows, q stored to q_out [rows][Hq][d]; k and
// v appended to the cache of every destination slot of the row
// (dst_slots[row_dst[r] + g], g < n_dst) at position row_pos[r]; a negative
// row_dst[r] names one slot, -(row_dst[r] + 1).
// qkv: `splits` fp32 split-K slices [splits][n_rows][(Hq + 2 Hkv) D] summed in
// order (splits <= 1: the finished projection)
hipError_t launch_rope_append(int dt, const float* qkv, int splits, int n_rows, const int32_t* row_pos,
                              const int32_t* row_dst, int n_dst, const int32_t* dst_slots,
                              const float* cs, int cs_stride, int Hq, int Hkv, int D,
                              const KvPages& kp, int layer,
                              void* q_out, void* kc, void* vc, hipStream_t s);

// ev_start / ev_stop (may be null): events stamped with the kernel's own
// start and end (attached to the dispatch, not recorded around it)
hipError_t launch_attention_bf16(const AttnItem* items, int n_items, const void* q,
                                 const void* kc, const void* vc, const KvPages& kp, int Hq, int Hkv,
                                 int D, int layer, void* out, float* part,
                                 hipStream_t s, hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr);

// Router logits [n][E] -> each row's top k experts and weights ([n][k]),
// then the n * k pairs grouped by expert (off [E + 1], pairs [n * k]).
hipError_t launch_moe_route(const float* logits, int n, int E, int k, int32_t* ids, float* w, int32_t* off,
                            int32_t* pairs, hipStream_t s);
// One grouped expert projection (epi: EPI_SWIGLU for gate|up, EPI_RESID for
// down, which writes routing-weighted planes).
hipError_t launch_moe_gemv(const MoeArgs& a, int epi, hipStream_t s);

// Most items one split block may have (bounds the combine's LDS).
constexpr int kMaxCombine = 64;

// blocks[b] = index of the first item of split block b.
hipError_t launch_attn_combine(const int32_t* blocks, int n_blocks, const AttnItem* items, const float* part,
                               int Hq, int Hkv, int D, void* out, hipStream_t s);

// Prefill / scoring attention tile: up to kPrefillWaves * (16 / G) consecutive
// query tokens of one sequence (workspace rows qrow0 .., positions pos0 ..)
// against every key they see, [0, pos0 + ntok), of one KV slot.
struct PrefillTile {
    int32_t qrow0;
    int32_t ntok;
    int32_t slot;
    int32_t pos0;
};
constexpr int kPrefillWaves = 8;

// One 4-wave workgroup per (tile, kv-head): each 32-position K/V step is
// loaded once into LDS and used by every wave (wave w takes the tile's tokens
// [w * 16/G, (w+1) * 16/G)); outputs are final (no split partials).
hipError_t launch_attention_prefill(const PrefillTile* tiles, int n_tiles, const void* q, const void* kc,
                                    const void* vc, const KvPages& kp, int Hq, int Hkv, int D, int layer,
                                    void* out, hipStream_t s);

// fp32 model dtype: one workgroup per (row, q-head), keys 0..row_pos[r].
hipError_t launch_attention_f32(int n_rows, const int32_t* row_slot, const int32_t* row_pos,
                                const float* q, const float* kc, const float* vc, const KvPages& kp,
                                int Hq, int Hkv, int D, int layer, float* out,
                                hipStream_t s);

// Per-chunk partial of the sampler (merged in chunk order by a second kernel).
struct SamplePart { float best_s; int best_v; float m; float s; };
constexpr int kSampleMaxChunks = 64;

// parts: [n][kSampleMaxChunks].
// Inference-stage log-probabilities: for logits row r < n_rows and every item
// k in [row_items[r], row_items[r+1]), out[item_idx[k]] = fl32(z_y / T) -
// LSE(fl32(z / T)) with y = targets[item_idx[k]] (NaN when y is outside
// [0, V)).  T > 0.
hipError_t launch_logprob(const float* logits, int ld, int n_rows, int V, const int32_t* row_items,
                          const int32_t* item_idx, const int32_t* targets, float T, float* out,
                          hipStream_t s);

// SampleParts a launch over n rows of V logits writes (0: a single chunk per
// row, no partials).
size_t sample_parts_needed(int n, int V);

// The sampler's allocation-free partial buffer: kStaticSampleParts entries
// in device memory of the current device (n * ceil(2048 / n) < 4096 for every
// n, so every launch fits).
constexpr int kStaticSampleParts = 4096;
hipError_t static_sample_parts(SamplePart** out);

hipError_t launch_sample(const float* logits, int ld, int n, int V, const int32_t* logit_row,
                         const uint64_t* uid, const int32_t* pos_new, const int32_t* forced,
                         uint64_t seed, float T, SamplePart* parts,
                         int32_t* out_tok, float* out_logp, hipStream_t s);

// Copy the live K/V of n slots between the pool and a packed staging buffer
// (dir 0: pool -> stage, dir 1: stage -> pool).  Slot i (lens[i] positions)
// starts at byte base[i] of the stage: for layer l, kv-head h (index
// l*Hkv + h): lens[i] K rows of rowbytes, then ceil8(lens[i]) / 8 V blocks of
// 8 * rowbytes (the pool's own layouts, page after page).  rowbytes =
// head_dim * es, es = element size.
hipError_t launch_kv_pack(int dir, const int32_t* slots, const int32_t* lens, const int64_t* base, int n, int L,
                          const KvPages& kp, int Hkv, int rowbytes, int es, void* kslab, void* vslab,
                          void* stage, hipStream_t s);

hipError_t launch_copy16(void* dst, const void* src, size_t n16, hipStream_t s);
// read-only stream of n16 16-byte words by n_blocks workgroups; out[b] = XOR of workgroup b's words
hipError_t launch_read16(const void* src, size_t n16, uint32_t* out, int n_blocks, hipStream_t s);
// n_blocks workgroups of four waves, each wave iters x 8 MFMA 32x32x16 bf16; out [n_blocks * 4]
hipError_t launch_mfma_probe(int n_blocks, int iters, float* out, hipStream_t s);

// Sampler noise-bound check over words [lo, lo + count): per workgroup, the
// number of violated bounds and the smallest margin of the fp32 bound.
hipError_t launch_gumbel_bound_probe(uint32_t lo, uint64_t count, int n_blocks, uint32_t* viol,
                                     float* min_margin, hipStream_t s);

}  // namespace rl
