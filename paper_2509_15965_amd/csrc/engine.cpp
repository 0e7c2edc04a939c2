// engine.cpp -- host side of the rollout decode library: argument validation,
// workspace layout, per-call index metadata, split-KV planning and kernel
// sequencing on the caller's stream.  Implements include/rl_decode.h.
#include "rl_decode.h"
#include "rl_internal.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <functional>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>
#include <unordered_map>
#include <vector>

using namespace rl;

namespace {

constexpr uint32_t kMagic = 0x524C4443u;   // "RLDC"
constexpr uint32_t kDead = 0xDEADDEADu;
constexpr int kStages = 3;                  // pinned metadata staging ring
constexpr int kPartItems = 8192;            // split-KV partial slots per call
constexpr int kAttnWaveTarget = 1024;       // split-KV: keep about one wave per SIMD, each as long as possible
constexpr int kSharedDecodeChunk = 256;     // split-KV keys per item in decode steps that read shared prompts
constexpr int kPrefillChunk = 1024;         // default keys per prefill work item
constexpr int kNoAllocMaxRows = 1 << 20;    // rows of one rl_sample_logits_noalloc call

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }
int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Bytes from one K (or V) block of a paged pool to the next: the page's rows
// rounded up to an odd number of 256-byte granules, so that no two blocks are
// a power of two apart (the decode attention's work items start at the same
// page offsets together; pages of 64 positions ran the 7B rollout's
// attention 6% faster padded than not).
size_t paged_block_bytes(size_t rows_bytes) {
    const size_t g = 256;
    size_t n = (rows_bytes + g - 1) / g;
    if (n % 2 == 0) ++n;
    return n * g;
}

struct Layout {
    int es = 0, cap = 0, R = 0, nqkv = 0, items_cap = 0;
    int page = 0, pages = 0, maxp = 1;   // K/V pages: positions each, pool size, table row length
    size_t block = 0;                    // elements from one (layer, page, kv-head) K/V block to the next
    size_t kv_bytes = 0, ws_bytes = 0;
    size_t off_x = 0, off_h = 0, off_qkv = 0, off_q = 0, off_attn = 0, off_mlp = 0;
    size_t off_part = 0, off_apart = 0, off_logits = 0, off_rope = 0, off_meta = 0;
    size_t off_spart = 0, off_tok = 0;
    size_t off_stage = 0, stage_bytes = 0;   // KV offload staging: the activation buffers x .. split-K partials
    size_t part_floats = 0, apart_floats = 0, meta_bytes = 0;
    // mixture of experts: router logits [R][E] fp32, per pair its expert and
    // weight, the pairs grouped by expert and each expert's range, the
    // pairs' SwiGLU rows [R*k][Fe] and their weighted outputs [k][R][H] fp32
    size_t off_router = 0, off_moe_ids = 0, off_moe_w = 0, off_moe_pairs = 0, off_moe_off = 0;
    size_t off_moe_act = 0, off_moe_out = 0;
};

bool cfg_check(const rl_model_config* c, rl_status* code, std::string* why) {
    auto bad = [&](rl_status s, const char* m) { *code = s; *why = m; return false; };
    if (!c) return bad(RL_ERR_INVALID_ARG, "config is NULL");
    if (c->reserved != 0) return bad(RL_ERR_INVALID_ARG, "config.reserved must be 0");
    if (c->kv_page_size != 0 &&
        (c->kv_page_size < 32 || c->kv_page_size > 65536 || c->kv_page_size % 32 != 0))
        return bad(RL_ERR_INVALID_ARG, "kv_page_size must be 0 or a multiple of 32 in [32, 65536]");
    if (c->kv_pages < 0 || (c->kv_page_size == 0 && c->kv_pages != 0) || c->kv_pages > (1 << 26))
        return bad(RL_ERR_INVALID_ARG, "kv_pages must be >= 0, and 0 without pages");
    if (c->n_layers < 1 || c->n_layers > 4096) return bad(RL_ERR_INVALID_ARG, "n_layers out of range");
    if (c->hidden < 8 || c->hidden > (1 << 16)) return bad(RL_ERR_INVALID_ARG, "hidden out of range");
    if (c->n_q_heads < 1 || c->n_kv_heads < 1 || c->n_q_heads > 1024) return bad(RL_ERR_INVALID_ARG, "head counts out of range");
    if ((c->n_experts == 0 && c->ffn < 8) || c->ffn < 0 || c->ffn > (1 << 20))
        return bad(RL_ERR_INVALID_ARG, "ffn out of range");   // a mixture of experts does not use it
    if (c->vocab < 8 || c->vocab > (1 << 24)) return bad(RL_ERR_INVALID_ARG, "vocab out of range");
    if (c->dtype != RL_DTYPE_FP32 && c->dtype != RL_DTYPE_BF16) return bad(RL_ERR_INVALID_ARG, "unknown dtype");
    if (!(c->rms_eps > 0.0) || !std::isfinite(c->rms_eps)) return bad(RL_ERR_INVALID_ARG, "rms_eps must be > 0");
    if (!(c->rope_theta > 1.0) || !std::isfinite(c->rope_theta)) return bad(RL_ERR_INVALID_ARG, "rope_theta must be > 1");
    if (c->max_seqs < 1 || c->max_seqs > (1 << 16)) return bad(RL_ERR_INVALID_ARG, "max_seqs out of range");
    if (c->max_ctx < 2 || c->max_ctx > (1 << 20)) return bad(RL_ERR_INVALID_ARG, "max_ctx out of range");
    if (c->max_prefill_tokens < 1 || c->max_prefill_tokens > (1 << 22)) return bad(RL_ERR_INVALID_ARG, "max_prefill_tokens out of range");
    if (c->head_dim != 64 && c->head_dim != 128) return bad(RL_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
    if (c->n_q_heads % c->n_kv_heads != 0) return bad(RL_ERR_UNSUPPORTED, "n_q_heads must be a multiple of n_kv_heads");
    if (c->n_q_heads / c->n_kv_heads > 16) return bad(RL_ERR_UNSUPPORTED, "more than 16 q-heads per kv-head");
    if (c->hidden % 8 || c->ffn % 8 || c->vocab % 8) return bad(RL_ERR_UNSUPPORTED, "hidden, ffn and vocab must be multiples of 8");
    if (c->dtype == RL_DTYPE_BF16) {
        // the bf16 GEMM kernels address a weight matrix with 32-bit byte offsets
        const uint64_t H = static_cast<uint64_t>(c->hidden), F = static_cast<uint64_t>(c->ffn);
        const uint64_t qkv = static_cast<uint64_t>(c->n_q_heads + 2 * c->n_kv_heads) * c->head_dim;
        const uint64_t widest = std::max({static_cast<uint64_t>(c->vocab) * H, 2 * F * H, qkv * H, H * F,
                                          H * static_cast<uint64_t>(c->n_q_heads) * c->head_dim});
        if (2 * widest > 0xFFFFFFFFull) return bad(RL_ERR_UNSUPPORTED, "a bf16 weight matrix spans 4 GiB or more");
    }
    if (c->n_experts != 0 || c->top_k != 0 || c->expert_ffn != 0) {
        if (c->n_experts < 1 || c->n_experts > kMoeMaxExperts) return bad(RL_ERR_INVALID_ARG, "n_experts out of range");
        if (c->top_k < 1 || c->top_k > std::min(c->n_experts, kMoeMaxTopK))
            return bad(RL_ERR_INVALID_ARG, "top_k must be in [1, min(n_experts, 16)]");
        if (c->expert_ffn < 16 || c->expert_ffn > (1 << 20) || c->expert_ffn % 16)
            return bad(RL_ERR_INVALID_ARG, "expert_ffn must be a positive multiple of 16");
        if (c->dtype != RL_DTYPE_BF16) return bad(RL_ERR_UNSUPPORTED, "mixture of experts needs bf16");
        if (c->hidden % 16 || c->hidden > 4096)
            return bad(RL_ERR_UNSUPPORTED, "mixture of experts needs hidden a multiple of 16 and <= 4096");
    }
    return true;
}

Layout make_layout(const rl_model_config& c) {
    Layout L;
    L.es = c.dtype == RL_DTYPE_BF16 ? 2 : 4;
    L.cap = static_cast<int>(align_up(static_cast<size_t>(c.max_ctx), 32));
    L.R = std::max(c.max_seqs, c.max_prefill_tokens);
    L.nqkv = (c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
    L.items_cap = std::max(kPartItems, L.R + c.max_seqs);
    const size_t es = L.es, R = L.R, H = c.hidden, F = c.ffn, V = c.vocab;
    const size_t HqD = static_cast<size_t>(c.n_q_heads) * c.head_dim;
    if (c.kv_page_size > 0) {
        L.page = c.kv_page_size;
        L.maxp = static_cast<int>((static_cast<size_t>(c.max_ctx) + L.page - 1) / L.page);
        L.pages = c.kv_pages > 0 ? c.kv_pages : c.max_seqs * L.maxp;
        L.block = paged_block_bytes(static_cast<size_t>(L.page) * c.head_dim * es) / es;
    } else {
        L.page = L.cap;
        L.maxp = 1;
        L.pages = c.max_seqs;
        L.block = static_cast<size_t>(L.cap) * c.head_dim;
    }
    L.kv_bytes = 2ull * c.n_layers * L.pages * c.n_kv_heads * L.block * es;
    L.part_floats = kPartCapFloats;
    if (c.dtype == RL_DTYPE_FP32) L.part_floats = std::max(L.part_floats, R * std::max(H, 2 * F));
    L.apart_floats = static_cast<size_t>(kPartItems) * c.n_kv_heads * 16 * (c.head_dim + 2);
    // per-row index arrays (position, KV destination, slot read, LM-head
    // selection, log-prob item offsets and targets), per-sequence arrays,
    // attention work items
    L.meta_bytes = 4 * (7 * R + 4 * static_cast<size_t>(c.max_seqs)) + 8 * static_cast<size_t>(c.max_seqs) +
                   sizeof(AttnItem) * static_cast<size_t>(L.items_cap) + 4096;
    // a paged pool's table travels with every call's metadata
    if (c.kv_page_size > 0) L.meta_bytes += 4 * static_cast<size_t>(c.max_seqs) * L.maxp + 16;
    size_t o = 0;
    auto take = [&](size_t bytes) { size_t r = o; o = align_up(o + bytes, 256); return r; };
    L.off_x = take(R * H * 4);
    L.off_h = take(R * H * es);
    L.off_qkv = take(R * L.nqkv * 4);
    L.off_q = take(R * HqD * es);
    L.off_attn = take(R * HqD * es);
    L.off_mlp = take(R * F * es);
    L.off_part = take(L.part_floats * 4);
    L.off_stage = L.off_x;
    L.stage_bytes = o - L.off_x;
    L.off_apart = take(L.apart_floats * 4);
    L.off_logits = take(static_cast<size_t>(c.max_seqs) * V * 4);
    L.off_rope = take(static_cast<size_t>(L.cap) * (c.head_dim / 2) * 2 * 4);
    L.off_meta = take(L.meta_bytes);
    L.off_tok = take(R * 4);   // packed token ids of a scoring pass
    L.off_spart = take(sizeof(SamplePart) * static_cast<size_t>(c.max_seqs) * kSampleMaxChunks);
    if (c.n_experts > 0) {
        const size_t E = c.n_experts, P = R * c.top_k, Fe = c.expert_ffn;
        L.off_router = take(R * E * 4);
        L.off_moe_ids = take(P * 4);
        L.off_moe_w = take(P * 4);
        L.off_moe_pairs = take(P * 4);
        L.off_moe_off = take((E + 1) * 4);
        L.off_moe_act = take(P * Fe * es);
        L.off_moe_out = take(P * H * 4);
    }
    L.ws_bytes = o;
    return L;
}

}  // namespace

struct rl_decode_ctx {
    uint32_t magic = kMagic;
    rl_model_config cfg{};
    rl_weights w{};
    Layout lay;
    uint8_t* kv = nullptr;
    uint8_t* ws = nullptr;
    hipStream_t stream = nullptr;
    int device = 0;
    std::vector<int32_t> len;
    // shared GRPO prompt: decode attention over positions [0, share_len[s])
    // of slot s reads slot share_src[s] (the group's first slot, holding the
    // same K/V); -1 = no sharing
    std::vector<int32_t> share_src, share_len;
    uint8_t* staging[kStages] = {nullptr, nullptr, nullptr};
    hipEvent_t stage_ev[kStages] = {nullptr, nullptr, nullptr};
    bool stage_used[kStages] = {false, false, false};
    int stage_next = 0;
    int64_t opt_chunk = 0;
    bool opt_shared = true;           // RL_OPT_SHARED_PREFIX
    bool opt_prefill_items = false;   // RL_OPT_PREFILL_ATTENTION = 1: split-KV work items
    int64_t opt_gemm = 0;             // RL_OPT_GEMM_PLAN
    uint32_t profile = 0;             // bit mask over kernel classes
    struct Pending { int kc; hipEvent_t a, b; };
    std::vector<Pending> pending;
    std::vector<hipEvent_t> ev_pool;
    rl_kernel_stats stats[RL_K_COUNT]{};
    rl_attn_plan_stats plan{};
    // measured GEMM plans (rl_decode_tune_gemms), sorted by (class, rows)
    struct TunedPlan { int kc, M, Nw, K, epi; GemmPlan p; float us; };
    std::vector<TunedPlan> tuned;
    std::string err;

    // K/V pages (kv_page_size > 0): per slot its pages in position order
    // (ptab[s * maxp + j], -1 = none; npages[s] of them), the free pages,
    // and per page the number of slots holding it (0 = free; the slots of a
    // GRPO group share the pages their prompt fills)
    std::vector<int32_t> ptab, npages, free_pages, pref;

    template <typename T> T* wsp(size_t off) const { return reinterpret_cast<T*>(ws + off); }
    uint8_t* kslab() const { return kv; }
    uint8_t* vslab() const { return kv + lay.kv_bytes / 2; }
    bool paged() const { return cfg.kv_page_size > 0; }
    // addressing of the contiguous pool, or of a paged one through a device copy of the table
    KvPages kvp(const int32_t* dev_table) const {
        return KvPages{paged() ? dev_table : nullptr, lay.maxp, lay.page, lay.pages, lay.block};
    }
    SamplePart* sample_parts() const { return reinterpret_cast<SamplePart*>(ws + lay.off_spart); }
    bool bf16() const { return cfg.dtype == RL_DTYPE_BF16; }
};

namespace {

const char* kClassNames[RL_K_COUNT] = {
    "embed", "rmsnorm", "gemm_qkv", "rope_append", "attention", "attn_combine", "gemm_o",
    "gemm_gate_up", "gemm_down", "gemm_lm_head", "splitk_reduce", "sample", "moe_route", "moe_experts"};

rl_status fail(rl_decode_ctx* c, rl_status s, const std::string& m) {
    if (c) c->err = m;
    return s;
}

rl_status hip_fail(rl_decode_ctx* c, hipError_t e, const char* where) {
    std::string m = std::string(where) + ": " + hipGetErrorString(e);
    return fail(c, RL_ERR_HIP, m);
}

bool ctx_ok(const rl_decode_ctx* c) { return c && c->magic == kMagic; }

// ---- profiling -----------------------------------------------------------
hipEvent_t get_event(rl_decode_ctx* c) {
    if (!c->ev_pool.empty()) { hipEvent_t e = c->ev_pool.back(); c->ev_pool.pop_back(); return e; }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

hipError_t harvest(rl_decode_ctx* c) {
    if (c->pending.empty()) return hipSuccess;
    hipError_t e = hipEventSynchronize(c->pending.back().b);
    if (e != hipSuccess) return e;
    for (auto& p : c->pending) {
        float ms = 0.0f;
        if (hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) c->stats[p.kc].total_ms += ms;
        c->ev_pool.push_back(p.a);
        c->ev_pool.push_back(p.b);
    }
    c->pending.clear();
    return hipSuccess;
}

// Launches of a class are counted (with their algorithmic bytes and FLOPs)
// and timed only while RL_OPT_PROFILE selects the class.
// Times one launch of a kernel class when RL_OPT_PROFILE selects it: an
// event pair recorded around the launch (which also spans the dispatch gap
// before the kernel starts), or, for a launch that takes them (attached),
// events stamped by the dispatch itself at the kernel's start and end.
struct Prof {
    rl_decode_ctx* c; int kc; hipEvent_t a = nullptr, b = nullptr; bool on = false, attached = false;
    Prof(rl_decode_ctx* c_, int kc_, bool attach = false) : c(c_), kc(kc_), attached(attach) {
        on = ((c->profile >> kc) & 1u) != 0;
        if (!on) return;
        a = get_event(c);
        if (attached) {
            b = get_event(c);
        } else if (a) {
            (void)hipEventRecord(a, c->stream);
        }
    }
    // events for a launch that stamps them itself (null when not profiled)
    hipEvent_t start() const { return attached && a && b ? a : nullptr; }
    hipEvent_t stop() const { return attached && a && b ? b : nullptr; }
    void done(double bytes, double flops) {
        if (!on) return;
        c->stats[kc].launches += 1;
        c->stats[kc].alg_bytes += bytes;
        c->stats[kc].alg_flops += flops;
        if (!attached && a) b = get_event(c);
        if (!a || !b) {
            if (a) c->ev_pool.push_back(a);
            if (b) c->ev_pool.push_back(b);
            return;
        }
        if (!attached) (void)hipEventRecord(b, c->stream);
        c->pending.push_back({kc, a, b});
        if (c->pending.size() >= 4096) (void)harvest(c);
    }
};

// ---- metadata staging ------------------------------------------------------
struct Meta {
    uint8_t* host; uint8_t* dev; size_t cap; size_t used = 0; bool overflow = false;
    template <typename T> T* take(size_t n, T** dptr) {
        used = align_up(used, 16);
        size_t bytes = n * sizeof(T);
        if (used + bytes > cap) { overflow = true; *dptr = nullptr; return nullptr; }
        T* h = reinterpret_cast<T*>(host + used);
        *dptr = reinterpret_cast<T*>(dev + used);
        used += bytes;
        return h;
    }
};

// ---- K/V pages --------------------------------------------------------------
int pages_for(const rl_decode_ctx* c, int len) { return (len + c->lay.page - 1) / c->lay.page; }

// Distinct slots with their final lengths (a later entry for a slot wins).
std::vector<std::pair<int, int>> final_lengths(int n, const int32_t* slots, const int32_t* lens) {
    std::vector<std::pair<int, int>> v;
    for (int i = 0; i < n; ++i) {
        bool found = false;
        for (auto& e : v)
            if (e.first == slots[i]) { e.second = lens[i]; found = true; }
        if (!found) v.emplace_back(slots[i], lens[i]);
    }
    return v;
}

// Pages freed by dropping, for each (slot, k), the slot's pages from index k
// on: those whose every holder is dropped.
int64_t pages_freed(const rl_decode_ctx* c, const std::vector<std::pair<int, int>>& drop) {
    const size_t mp = static_cast<size_t>(c->lay.maxp);
    std::unordered_map<int32_t, int> refs;
    for (const auto& d : drop)
        for (int j = d.second; j < c->npages[d.first]; ++j) ++refs[c->ptab[d.first * mp + j]];
    int64_t n = 0;
    for (const auto& e : refs) n += c->pref[e.first] == e.second;
    return n;
}

// Slot s keeps its first `keep` pages; a page nobody holds any more is free.
void drop_pages(rl_decode_ctx* c, int s, int keep, bool* freed) {
    const size_t mp = static_cast<size_t>(c->lay.maxp);
    while (c->npages[s] > keep) {
        int32_t& pg = c->ptab[s * mp + --c->npages[s]];
        if (--c->pref[pg] == 0) {
            c->free_pages.push_back(pg);
            *freed = true;
        }
        pg = -1;
    }
}

// lowest page first: a slab that has been filled and emptied again hands out
// neighbouring pages to the positions of one sequence, as a fresh one does
void sort_free(rl_decode_ctx* c) {
    std::sort(c->free_pages.begin(), c->free_pages.end(), std::greater<int32_t>());
}

int32_t take_page(rl_decode_ctx* c, int holders) {
    const int32_t pg = c->free_pages.back();
    c->free_pages.pop_back();
    c->pref[pg] = holders;
    return pg;
}

// Whether the slots can hold these lengths with the free pages (pages given
// back count).  fresh: the slots' pages are replaced from position 0 (their
// K/V is rewritten); otherwise each keeps the pages up to its new length.
// Always true for a contiguous pool.
bool pages_fit(const rl_decode_ctx* c, const std::vector<std::pair<int, int>>& want, bool fresh = false,
               int64_t extra = 0) {
    if (!c->paged()) return true;
    int64_t need = extra;
    std::vector<std::pair<int, int>> drop;
    for (const auto& e : want) {
        const int keep = fresh ? 0 : std::min(pages_for(c, e.second), c->npages[e.first]);
        drop.emplace_back(e.first, keep);
        need += pages_for(c, e.second) - keep;
    }
    return need <= static_cast<int64_t>(c->free_pages.size()) + pages_freed(c, drop);
}

// Give every slot exactly the pages its length needs (pages_fit held); new
// pages are the slot's own.
void set_pages(rl_decode_ctx* c, const std::vector<std::pair<int, int>>& want, bool fresh = false) {
    if (!c->paged()) return;
    bool freed = false;
    for (const auto& e : want) drop_pages(c, e.first, fresh ? 0 : pages_for(c, e.second), &freed);
    if (freed) sort_free(c);
    const size_t mp = static_cast<size_t>(c->lay.maxp);
    for (const auto& e : want) {
        const int s = e.first, need = pages_for(c, e.second);
        while (c->npages[s] < need) c->ptab[s * mp + c->npages[s]++] = take_page(c, 1);
    }
}

// Index of the page holding position len of slot s when len ends inside a
// page that other slots also hold, else -1.
int shared_tail_page(const rl_decode_ctx* c, int s, int len) {
    if (!c->paged() || len % c->lay.page == 0) return -1;
    const int j = len / c->lay.page;
    if (j >= c->npages[s]) return -1;
    return c->pref[c->ptab[s * static_cast<size_t>(c->lay.maxp) + j]] > 1 ? j : -1;
}

// Copy page `from` into page `to`: every layer's and kv-head's K and V block.
hipError_t copy_page(rl_decode_ctx* c, int32_t from, int32_t to) {
    const Layout& L = c->lay;
    const size_t pitch = L.block * L.es;
    const size_t rows = static_cast<size_t>(L.page) * c->cfg.head_dim * L.es;
    const size_t Hkv = static_cast<size_t>(c->cfg.n_kv_heads);
    for (int v = 0; v < 2; ++v) {
        uint8_t* slab = v ? c->vslab() : c->kslab();
        for (int l = 0; l < c->cfg.n_layers; ++l) {
            const uint8_t* src = slab + (static_cast<size_t>(l) * L.pages + from) * Hkv * pitch;
            uint8_t* dst = slab + (static_cast<size_t>(l) * L.pages + to) * Hkv * pitch;
            const hipError_t e = hipMemcpy2DAsync(dst, pitch, src, pitch, rows, Hkv, hipMemcpyDeviceToDevice,
                                                  c->stream);
            if (e != hipSuccess) return e;
        }
    }
    return hipSuccess;
}

// Pages of a group's prompt that the group shares: the ones it fills (0 for
// a contiguous pool).  Prefill and scoring write those K/V rows once.
int shared_prompt_pages(const rl_decode_ctx* c, int plen) { return c->paged() ? plen / c->lay.page : 0; }

// Pages for a call that writes each slot's K/V from position 0: slot
// slots[g * group + k] holds prompt g (plen[g] positions, its full pages
// shared by the group) and then its own positions up to lens[g * group + k].
bool group_pages_fit(const rl_decode_ctx* c, int n_prompts, int group, const int32_t* slots,
                     const std::vector<int>& plen, const std::vector<int32_t>& lens) {
    if (!c->paged()) return true;
    int64_t need = 0;
    std::vector<std::pair<int, int>> drop;
    for (int g = 0; g < n_prompts; ++g) {
        const int sh = shared_prompt_pages(c, plen[g]);
        need += sh;
        for (int k = 0; k < group; ++k) {
            const int i = g * group + k;
            drop.emplace_back(slots[i], 0);
            need += pages_for(c, lens[i]) - sh;
        }
    }
    return need <= static_cast<int64_t>(c->free_pages.size()) + pages_freed(c, drop);
}

void set_group_pages(rl_decode_ctx* c, int n_prompts, int group, const int32_t* slots,
                     const std::vector<int>& plen, const std::vector<int32_t>& lens) {
    if (!c->paged()) return;
    bool freed = false;
    for (int i = 0; i < n_prompts * group; ++i) drop_pages(c, slots[i], 0, &freed);
    if (freed) sort_free(c);
    const size_t mp = static_cast<size_t>(c->lay.maxp);
    for (int g = 0; g < n_prompts; ++g) {
        const int sh = shared_prompt_pages(c, plen[g]);
        for (int j = 0; j < sh; ++j) {
            const int32_t pg = take_page(c, group);
            for (int k = 0; k < group; ++k) c->ptab[slots[g * group + k] * mp + j] = pg;
        }
        for (int k = 0; k < group; ++k) {
            const int i = g * group + k, s = slots[i];
            c->npages[s] = sh;
            while (c->npages[s] < pages_for(c, lens[i])) c->ptab[s * mp + c->npages[s]++] = take_page(c, 1);
        }
    }
}

// A paged pool's table region in this call's metadata (taken with the other
// arrays, filled once the call's pages are set).
struct PageStage { int32_t* host = nullptr; int32_t* dev = nullptr; };

PageStage take_pages(rl_decode_ctx* c, Meta* m) {
    PageStage ps;
    if (c->paged()) ps.host = m->take<int32_t>(c->ptab.size(), &ps.dev);
    return ps;
}

KvPages fill_pages(rl_decode_ctx* c, const PageStage& ps) {
    if (c->paged() && ps.host) std::memcpy(ps.host, c->ptab.data(), c->ptab.size() * sizeof(int32_t));
    return c->kvp(ps.dev);
}

rl_status begin_meta(rl_decode_ctx* c, Meta* m, int* stage) {
    int s = c->stage_next;
    if (c->stage_used[s]) {
        hipError_t e = hipEventSynchronize(c->stage_ev[s]);
        if (e != hipSuccess) return hip_fail(c, e, "staging wait");
    }
    *stage = s;
    m->host = c->staging[s];
    m->dev = c->ws + c->lay.off_meta;
    m->cap = c->lay.meta_bytes;
    m->used = 0;
    return RL_OK;
}

rl_status upload_meta(rl_decode_ctx* c, Meta* m, int stage) {
    if (m->overflow) return fail(c, RL_ERR_CAPACITY, "per-call metadata exceeds its workspace region");
    hipError_t e = hipMemcpyAsync(m->dev, m->host, m->used, hipMemcpyHostToDevice, c->stream);
    if (e != hipSuccess) return hip_fail(c, e, "metadata upload");
    e = hipEventRecord(c->stage_ev[stage], c->stream);
    if (e != hipSuccess) return hip_fail(c, e, "metadata event");
    c->stage_used[stage] = true;
    c->stage_next = (stage + 1) % kStages;
    return RL_OK;
}

// ---- forward pass description ----------------------------------------------
struct Fwd {
    KvPages kvp{nullptr, 1, 0, 0, 0};          // K/V addressing of this call
    int rows = 0;
    const int32_t* tok = nullptr;
    const void* embeds = nullptr;
    int n_embed_rows = 0;
    const int32_t* row_pos = nullptr;
    const int32_t* row_dst = nullptr;
    int n_dst = 1;
    const int32_t* dst_slots = nullptr;
    const int32_t* row_slot = nullptr;      // fp32 attention: slot each row reads
    const AttnItem* items = nullptr;
    int n_items = 0;
    int n_partial_items = 0;
    const PrefillTile* tiles = nullptr;     // prefill / scoring: shared-LDS tiles instead of items
    int n_tiles = 0;
    const int32_t* split_blocks = nullptr;   // first item of every split block
    int n_split_blocks = 0;
    // decode attention plan (build_items): work items, those over a shared
    // prompt chunk, pair items, workgroups staging a shared chunk in LDS
    int plan_items = 0, plan_shared = 0, plan_pairs = 0, plan_lds = 0;
    double attn_kv_positions = 0;           // algorithmic KV positions read per kv-head
    double attn_score_positions = 0;        // sum over rows of keys attended
    const int32_t* final_sel = nullptr;     // rows fed to the LM head (nullptr: all)
    int n_final = 0;
    float* logits = nullptr;
    int n_out = 0;
    const int32_t* logit_row = nullptr;
    const uint64_t* uid = nullptr;
    const int32_t* pos_new = nullptr;
    const int32_t* forced = nullptr;
    uint64_t seed = 0;
    float T = 1.0f;
    int32_t* out_tok = nullptr;
    float* out_logp = nullptr;
    // scoring pass (inference stage): instead of sampling, log-probabilities
    // of given tokens for the LM-head rows; row i of final_sel owns items
    // [score_items[i], score_items[i+1]) of score_idx, each an index into
    // score_targets and out_logp
    const int32_t* score_items = nullptr;
    const int32_t* score_idx = nullptr;
    const int32_t* score_targets = nullptr;
    int score_chunk = 0;                    // LM-head rows per chunk (rows of f.logits)
};

// Y = A . W^T with the given epilogue.  When the plan splits K, fp32 partials
// land in the split-K buffer: SwiGLU and plain fp32 outputs are reduced here;
// with `defer` set (q|k|v and residual projections) *splits reports the slice
// count and the caller reduces.  A residual GEMM with one split adds into x
// directly (bf16); the fp32 model always goes through the partial buffer.
// The measured plan of the smallest tuned batch size >= M for this class and
// GEMM shape (false: none tuned).
bool tuned_plan(const rl_decode_ctx* c, int kc, int M, int Nw, int K, int epi, GemmPlan* p, float* us) {
    for (const auto& t : c->tuned) {
        if (t.kc != kc || t.Nw != Nw || t.K != K || t.epi != epi || t.M < M) continue;
        *p = t.p;
        if (us) *us = t.us;
        return true;   // sorted by rows: the first match is the smallest
    }
    return false;
}

// Plan of a bf16 GEMM: the RL_OPT_GEMM_PLAN override when it can serve this
// GEMM, else the measured plan, else the cost model.
GemmPlan choose_plan(const rl_decode_ctx* c, int kc, int M, int Nw, int K, int epi) {
    GemmPlan p;
    const int F = c->cfg.ffn;
    if (c->opt_gemm != 0 && plan_gemm_forced(M, Nw, K, epi, F, c->opt_gemm, &p)) return p;
    if (tuned_plan(c, kc, M, Nw, K, epi, &p, nullptr)) return p;
    return plan_gemm_bf16(M, Nw, K, epi, F);
}

rl_status run_gemm_plan(rl_decode_ctx* c, int kc, const GemmPlan* plan, const void* A, int lda, const void* W,
                        int M, int Nw, int K, int epi, float* out_f32, int ldo, float* resid, int ldr, void* act,
                        int ld_act, bool defer, int* splits);

rl_status run_gemm(rl_decode_ctx* c, int kc, const void* A, int lda, const void* W, int M, int Nw,
                   int K, int epi, float* out_f32, int ldo, float* resid, int ldr, void* act,
                   int ld_act, bool defer, int* splits) {
    return run_gemm_plan(c, kc, nullptr, A, lda, W, M, Nw, K, epi, out_f32, ldo, resid, ldr, act, ld_act, defer,
                         splits);
}

// run_gemm with a given plan (nullptr: choose_plan's)
rl_status run_gemm_plan(rl_decode_ctx* c, int kc, const GemmPlan* plan, const void* A, int lda, const void* W,
                        int M, int Nw, int K, int epi, float* out_f32, int ldo, float* resid, int ldr, void* act,
                        int ld_act, bool defer, int* splits) {
    const rl_model_config& cf = c->cfg;
    GemmArgs a{};
    a.A = A; a.lda = lda; a.W = W; a.ldw = K; a.M = M; a.Nw = Nw; a.K = K; a.epi = epi;
    a.out_f32 = out_f32; a.ldo = ldo; a.resid = resid; a.ldr = ldr; a.act = act; a.ld_act = ld_act;
    a.F = cf.ffn;
    a.partial = c->wsp<float>(c->lay.off_part);
    const double es = c->lay.es;
    const int n_out = epi == EPI_SWIGLU ? cf.ffn : Nw;
    double out_bytes = epi == EPI_F32 ? 4.0 * M * n_out : epi == EPI_RESID ? 8.0 * M * n_out : es * M * n_out;
    double bytes = es * Nw * K + es * M * K + out_bytes;
    double flops = 2.0 * M * Nw * K;
    hipError_t e;
    *splits = 0;
    if (c->bf16()) {
        const GemmPlan p = plan ? *plan : choose_plan(c, kc, M, Nw, K, epi);
        {
            Prof pr(c, kc);
            e = launch_gemm_bf16(a, p, c->stream);
            if (e != hipSuccess) return hip_fail(c, e, "gemm launch");
            pr.done(bytes, flops);
        }
        if (p.splits > 1) {
            if (defer) {
                *splits = p.splits;
                return RL_OK;
            }
            Prof pr(c, RL_K_SPLITK_REDUCE);
            e = launch_splitk_reduce(DT_BF16, a, p.splits, a.partial, c->stream);
            if (e != hipSuccess) return hip_fail(c, e, "split-K reduce launch");
            pr.done(4.0 * p.splits * M * Nw + out_bytes, 0.0);
        }
        return RL_OK;
    }
    GemmArgs g = a;
    if (epi != EPI_F32) { g.out_f32 = a.partial; g.ldo = Nw; }
    {
        Prof pr(c, kc);
        e = launch_gemm_f32(g, c->stream);
        if (e != hipSuccess) return hip_fail(c, e, "gemm launch");
        pr.done(bytes, flops);
    }
    if (epi == EPI_RESID && defer) {
        *splits = 1;
        return RL_OK;
    }
    if (epi != EPI_F32) {
        Prof pr(c, RL_K_SPLITK_REDUCE);
        e = launch_splitk_reduce(DT_F32, a, 1, a.partial, c->stream);
        if (e != hipSuccess) return hip_fail(c, e, "epilogue launch");
        pr.done(4.0 * M * Nw + out_bytes, 0.0);
    }
    return RL_OK;
}

// Sum `splits` fp32 slices of the split-K buffer (fixed order) into out (F32)
// or into the residual x (RESID), spread over many workgroups.
rl_status reduce_splits(rl_decode_ctx* c, int epi, int M, int N, int splits, float* out, int ldo, float* resid) {
    GemmArgs a{};
    a.M = M; a.Nw = N; a.epi = epi; a.out_f32 = out; a.ldo = ldo; a.resid = resid; a.ldr = N; a.F = c->cfg.ffn;
    Prof pr(c, RL_K_SPLITK_REDUCE);
    hipError_t e = launch_splitk_reduce(c->bf16() ? DT_BF16 : DT_F32, a, splits, c->wsp<float>(c->lay.off_part),
                                        c->stream);
    if (e != hipSuccess) return hip_fail(c, e, "split-K reduce launch");
    pr.done(4.0 * splits * M * N + (epi == EPI_RESID ? 8.0 : 4.0) * M * N, 0.0);
    return RL_OK;
}

// x += the split-K slices of a deferred RESID GEMM (splits > 0), then
// h = rmsnorm(x) * g in one fused pass per row: at any batch size when a row
// fits one float4 per thread (H <= 4096), else from kResidNormMinRows rows
// (enough rows to hide the grouped loads); below, the wide reduction and the norm.
constexpr int kResidNormMinRows = 64;
// part: the slices to add (default: the split-K partials region); a mixture
// of experts passes its weighted expert outputs (one plane per choice, H <= 4096).
rl_status resid_then_norm(rl_decode_ctx* c, int dt, int splits, float* x, int n, int H, const void* g, float eps,
                          void* h, const float* part = nullptr) {
    const double es = c->lay.es;
    hipError_t e;
    if (splits > 0 && H % 4 == 0 && (H <= 4096 || (n >= kResidNormMinRows && H <= 8192))) {
        Prof pr(c, RL_K_SPLITK_REDUCE);
        e = launch_resid_norm(dt, part ? part : c->wsp<float>(c->lay.off_part), splits, x, n, H, g, eps, h,
                              c->stream);
        if (e != hipSuccess) return hip_fail(c, e, "residual + rmsnorm launch");
        pr.done(n * H * (4.0 * splits + 8.0 + es) + H * es, 0.0);
        return RL_OK;
    }
    if (splits > 0) {
        rl_status st = reduce_splits(c, EPI_RESID, n, H, splits, nullptr, 0, x);
        if (st != RL_OK) return st;
    }
    Prof pr(c, RL_K_RMSNORM);
    e = launch_rmsnorm(dt, x, nullptr, n, H, g, eps, h, c->stream);
    if (e != hipSuccess) return hip_fail(c, e, "rmsnorm launch");
    pr.done(n * H * (4.0 + es) + H * es, 0.0);
    return RL_OK;
}

// Mixture-of-experts MLP of layer l over n rows of h: router logits, top-k
// and grouping, then the experts' gate|up (SwiGLU) and down projections,
// whose routing-weighted outputs land in k planes of [n][H] fp32.
rl_status run_moe(rl_decode_ctx* c, int l, int n, const void* h) {
    const rl_model_config& cf = c->cfg;
    const Layout& L = c->lay;
    const int H = cf.hidden, E = cf.n_experts, k = cf.top_k, Fe = cf.expert_ffn;
    const size_t esz = static_cast<size_t>(L.es);
    const uint8_t* wr = static_cast<const uint8_t*>(c->w.w_router) + static_cast<size_t>(l) * E * H * esz;
    float* logits = c->wsp<float>(L.off_router);
    int splits = 0;
    rl_status st = run_gemm(c, RL_K_MOE_ROUTE, h, H, wr, n, E, H, EPI_F32, logits, E, nullptr, 0, nullptr, 0, false,
                            &splits);   // split-K slices, if any, are summed inside (not deferred)
    if (st != RL_OK) return st;
    int32_t* ids = c->wsp<int32_t>(L.off_moe_ids);
    float* pw = c->wsp<float>(L.off_moe_w);
    int32_t* pairs = c->wsp<int32_t>(L.off_moe_pairs);
    int32_t* off = c->wsp<int32_t>(L.off_moe_off);
    hipError_t e;
    {
        Prof pr(c, RL_K_MOE_ROUTE);
        e = launch_moe_route(logits, n, E, k, ids, pw, off, pairs, c->stream);
        if (e != hipSuccess) return hip_fail(c, e, "expert routing launch");
        pr.done(n * (E * 4.0 + k * 12.0), 0.0);
    }
    MoeArgs a{};
    a.E = E; a.k = k; a.n_rows = n; a.npairs = n * k;
    a.off = off; a.pairs = pairs; a.pw = pw;
    {
        Prof pr(c, RL_K_MOE_EXPERTS);
        MoeArgs g = a;   // gate|up: token rows -> SwiGLU rows of the pairs
        g.A = static_cast<const uint16_t*>(h); g.lda = H;
        g.W = static_cast<const uint16_t*>(c->w.w_exp_gate_up) + static_cast<size_t>(l) * E * 2 * Fe * H;
        g.w_expert = static_cast<size_t>(2) * Fe * H; g.ldw = H; g.K = H; g.Nw = 2 * Fe; g.F = Fe;
        g.groups = (Fe + kMoeRowsPerGroup / 2 - 1) / (kMoeRowsPerGroup / 2);
        g.act = reinterpret_cast<uint16_t*>(c->ws + L.off_moe_act); g.ld_act = Fe;
        e = launch_moe_gemv(g, EPI_SWIGLU, c->stream);
        if (e != hipSuccess) return hip_fail(c, e, "expert gate|up launch");
        MoeArgs d = a;   // down: SwiGLU rows -> weighted output planes
        d.A = g.act; d.lda = Fe;
        d.W = static_cast<const uint16_t*>(c->w.w_exp_down) + static_cast<size_t>(l) * E * H * Fe;
        d.w_expert = static_cast<size_t>(H) * Fe; d.ldw = Fe; d.K = Fe; d.Nw = H; d.F = 0;
        d.groups = (H + kMoeRowsPerGroup - 1) / kMoeRowsPerGroup;
        d.plane = c->wsp<float>(L.off_moe_out);
        e = launch_moe_gemv(d, EPI_RESID, c->stream);
        if (e != hipSuccess) return hip_fail(c, e, "expert down launch");
        // bytes: the experts that can be reached (at most n * k of E) and the pairs' rows
        const double reach = std::min<double>(E, static_cast<double>(n) * k);
        pr.done(reach * 3.0 * H * Fe * L.es + n * k * (2.0 * Fe * L.es + H * 4.0) + n * H * L.es,
                2.0 * n * k * 3.0 * H * Fe);
    }
    return RL_OK;
}

rl_status run_forward(rl_decode_ctx* c, const Fwd& f) {
    const rl_model_config& cf = c->cfg;
    const Layout& L = c->lay;
    const int dt = c->bf16() ? DT_BF16 : DT_F32;
    const int H = cf.hidden, Hq = cf.n_q_heads, Hkv = cf.n_kv_heads, D = cf.head_dim, F = cf.ffn;
    const int HqD = Hq * D;
    const double es = L.es;
    const float eps = static_cast<float>(cf.rms_eps);
    float* x = c->wsp<float>(L.off_x);
    void* h = c->ws + L.off_h;
    float* qkv = c->wsp<float>(L.off_qkv);
    void* q = c->ws + L.off_q;
    void* attn = c->ws + L.off_attn;
    void* mlp = c->ws + L.off_mlp;
    float* apart = c->wsp<float>(L.off_apart);
    const float* cs = c->wsp<float>(L.off_rope);
    const int cs_stride = L.cap * (D / 2);
    hipError_t e;
    const int n = f.rows;
    const size_t esz = static_cast<size_t>(L.es);
    auto lw = [&](const void* base, int l, size_t per_layer) {
        return static_cast<const uint8_t*>(base) + static_cast<size_t>(l) * per_layer * esz;
    };


    {   // embedding, fused with the first layer's attention norm
        Prof pr(c, RL_K_EMBED);
        e = launch_embed(dt, f.tok, n, c->w.embed, cf.vocab, f.embeds, f.n_embed_rows, H, x,
                         c->w.attn_norm, eps, h, c->stream);
        if (e != hipSuccess) return hip_fail(c, e, "embed launch");
        pr.done(n * H * (2.0 * es + 4.0), 0.0);
    }
    for (int l = 0; l < cf.n_layers; ++l) {
        const uint8_t* wqkv = lw(c->w.w_qkv, l, static_cast<size_t>(L.nqkv) * H);
        const uint8_t* wo = lw(c->w.w_o, l, static_cast<size_t>(H) * HqD);
        const uint8_t* mn = lw(c->w.mlp_norm, l, H);
        const bool moe = cf.n_experts > 0;   // no dense MLP weights then
        const uint8_t* wgu = moe ? nullptr : lw(c->w.w_gate_up, l, static_cast<size_t>(2) * F * H);
        const uint8_t* wd = moe ? nullptr : lw(c->w.w_down, l, static_cast<size_t>(H) * F);
        const bool last_layer = l + 1 == cf.n_layers;
        // norm applied after this layer's down projection: the next layer's
        // attention norm, or the final norm (all rows; prefill selects rows later)
        const void* next_norm = last_layer ? c->w.final_norm : static_cast<const void*>(lw(c->w.attn_norm, l + 1, H));
        const bool norm_after_down = !last_layer || f.final_sel == nullptr;

        int splits = 0;
        rl_status st = run_gemm(c, RL_K_GEMM_QKV, h, H, wqkv, n, L.nqkv, H, EPI_F32, qkv, L.nqkv,
                                nullptr, 0, nullptr, 0, true, &splits);
        if (st != RL_OK) return st;
        {   // RoPE + KV append; with split K it sums the fp32 slices itself
            const int qs = splits > 1 ? splits : 1;
            const float* src = splits > 1 ? c->wsp<float>(L.off_part) : qkv;
            Prof pr(c, RL_K_ROPE_APPEND);
            e = launch_rope_append(dt, src, qs, n, f.row_pos, f.row_dst, f.n_dst, f.dst_slots, cs, cs_stride, Hq,
                                   Hkv, D, f.kvp, l, q, c->kslab(), c->vslab(), c->stream);
            if (e != hipSuccess) return hip_fail(c, e, "rope/append launch");
            pr.done(n * (qs * L.nqkv * 4.0 + HqD * es + f.n_dst * 2.0 * Hkv * D * es), 0.0);
        }
        {
            Prof pr(c, RL_K_ATTENTION, c->bf16() && !f.tiles);
            if (c->bf16() && f.tiles)
                e = launch_attention_prefill(f.tiles, f.n_tiles, q, c->kslab(), c->vslab(), f.kvp, Hq, Hkv, D,
                                             l, attn, c->stream);
            else if (c->bf16())
                e = launch_attention_bf16(f.items, f.n_items, q, c->kslab(), c->vslab(), f.kvp, Hq, Hkv,
                                          D, l, attn, apart, c->stream, pr.start(), pr.stop());
            else
                e = launch_attention_f32(n, f.row_slot, f.row_pos, static_cast<const float*>(q),
                                         reinterpret_cast<const float*>(c->kslab()),
                                         reinterpret_cast<const float*>(c->vslab()), f.kvp, Hq, Hkv, D,
                                         l, static_cast<float*>(attn), c->stream);
            if (e != hipSuccess) return hip_fail(c, e, "attention launch");
            pr.done(f.attn_kv_positions * Hkv * 2.0 * D * es + 2.0 * n * HqD * es,
                    4.0 * Hq * D * f.attn_score_positions);
        }
        if (f.n_split_blocks > 0) {
            Prof pr(c, RL_K_ATTN_COMBINE);
            e = launch_attn_combine(f.split_blocks, f.n_split_blocks, f.items, apart, Hq, Hkv, D, attn, c->stream);
            if (e != hipSuccess) return hip_fail(c, e, "combine launch");
            pr.done(f.n_partial_items * 16.0 * Hkv * (D + 2) * 4.0, 0.0);
        }
        st = run_gemm(c, RL_K_GEMM_O, attn, HqD, wo, n, H, HqD, EPI_RESID, nullptr, 0, x, H, nullptr, 0,
                      true, &splits);
        if (st != RL_OK) return st;
        st = resid_then_norm(c, dt, splits, x, n, H, mn, eps, h);   // MLP norm
        if (st != RL_OK) return st;
        if (moe) {   // mixture of experts; its k weighted outputs are summed with the residual
            st = run_moe(c, l, n, h);
            if (st != RL_OK) return st;
            st = resid_then_norm(c, dt, cf.top_k, x, n, H, next_norm, eps, h, c->wsp<float>(L.off_moe_out));
            if (st != RL_OK) return st;
            continue;
        }
        st = run_gemm(c, RL_K_GEMM_GATE_UP, h, H, wgu, n, 2 * F, H, EPI_SWIGLU, nullptr, 0, nullptr, 0, mlp, F,
                      false, &splits);
        if (st != RL_OK) return st;
        st = run_gemm(c, RL_K_GEMM_DOWN, mlp, F, wd, n, H, F, EPI_RESID, nullptr, 0, x, H, nullptr, 0, true,
                      &splits);
        if (st != RL_OK) return st;
        if (norm_after_down) {   // next layer's attention norm, or the final norm (decode)
            st = resid_then_norm(c, dt, splits, x, n, H, next_norm, eps, h);
            if (st != RL_OK) return st;
        } else if (splits > 0) {
            st = reduce_splits(c, EPI_RESID, n, H, splits, nullptr, 0, x);
            if (st != RL_OK) return st;
        }
    }
    const int nf = f.final_sel ? f.n_final : n;
    if (f.final_sel) {   // prefill: final norm of each prompt's last row only
        Prof pr(c, RL_K_RMSNORM);
        e = launch_rmsnorm(dt, x, f.final_sel, nf, H, c->w.final_norm, eps, h, c->stream);
        if (e != hipSuccess) return hip_fail(c, e, "final rmsnorm launch");
        pr.done(nf * H * (4.0 + es) + H * es, 0.0);
    }
    if (f.score_items) {   // LM head and log-probabilities in chunks of score_chunk rows
        const int V = cf.vocab;
        for (int r0 = 0; r0 < nf; r0 += f.score_chunk) {
            const int nc = std::min(f.score_chunk, nf - r0);
            int sp = 0;
            const uint8_t* hr = static_cast<const uint8_t*>(h) + static_cast<size_t>(r0) * H * esz;
            rl_status st = run_gemm(c, RL_K_GEMM_LM_HEAD, hr, H, c->w.lm_head, nc, V, H, EPI_F32, f.logits, V,
                                    nullptr, 0, nullptr, 0, false, &sp);
            if (st != RL_OK) return st;
            Prof pr(c, RL_K_SAMPLE);
            e = launch_logprob(f.logits, V, nc, V, f.score_items + r0, f.score_idx, f.score_targets, f.T,
                               f.out_logp, c->stream);
            if (e != hipSuccess) return hip_fail(c, e, "log-prob launch");
            pr.done(nc * V * 4.0, 0.0);
        }
        return RL_OK;
    }
    int splits = 0;
    rl_status st = run_gemm(c, RL_K_GEMM_LM_HEAD, h, H, c->w.lm_head, nf, cf.vocab, H, EPI_F32, f.logits,
                            cf.vocab, nullptr, 0, nullptr, 0, false, &splits);
    if (st != RL_OK) return st;
    {
        Prof pr(c, RL_K_SAMPLE);
        e = launch_sample(f.logits, cf.vocab, f.n_out, cf.vocab, f.logit_row, f.uid, f.pos_new, f.forced,
                          f.seed, f.T, c->sample_parts(), f.out_tok, f.out_logp,
                          c->stream);
        if (e != hipSuccess) return hip_fail(c, e, "sample launch");
        pr.done(f.n_out * (cf.vocab * 4.0 + 8.0), 0.0);
    }
    return RL_OK;
}

// ---- GEMM plan measurement ------------------------------------------------
// One timed unit of a decode GEMM class at M rows on layer l: the GEMM with
// plan p, then the kernel that consumes its output as a decode step issues it
// (q|k|v: RoPE summing the split-K slices, with no K/V destination; o and
// down: residual sum + RMSNorm; gate-up and LM head: their split-K
// reduction).  Operands are the workspace's activation buffers; `zeros` holds
// M zero positions.
rl_status tune_unit(rl_decode_ctx* c, int kc, const GemmPlan& p, int M, int l, const int32_t* zeros) {
    const rl_model_config& cf = c->cfg;
    const Layout& L = c->lay;
    const int H = cf.hidden, Hq = cf.n_q_heads, Hkv = cf.n_kv_heads, D = cf.head_dim, F = cf.ffn;
    const int HqD = Hq * D;
    const size_t esz = static_cast<size_t>(L.es);
    auto lw = [&](const void* base, size_t per_layer) {
        return static_cast<const uint8_t*>(base) + static_cast<size_t>(l) * per_layer * esz;
    };
    float* x = c->wsp<float>(L.off_x);
    void* h = c->ws + L.off_h;
    float* qkv = c->wsp<float>(L.off_qkv);
    const float eps = static_cast<float>(cf.rms_eps);
    int splits = 0;
    rl_status st;
    switch (kc) {
        case RL_K_GEMM_QKV: {
            st = run_gemm_plan(c, kc, &p, h, H, lw(c->w.w_qkv, static_cast<size_t>(L.nqkv) * H), M, L.nqkv, H,
                               EPI_F32, qkv, L.nqkv, nullptr, 0, nullptr, 0, true, &splits);
            if (st != RL_OK) return st;
            const float* src = splits > 1 ? c->wsp<float>(L.off_part) : qkv;
            // no K/V destination (n_dst = 0), so the pool is not addressed
            const hipError_t e = launch_rope_append(DT_BF16, src, splits > 1 ? splits : 1, M, zeros, zeros, 0, nullptr,
                                                    c->wsp<float>(L.off_rope), L.cap * (D / 2), Hq, Hkv, D,
                                                    c->kvp(nullptr), l, c->ws + L.off_q, c->kslab(), c->vslab(),
                                                    c->stream);
            return e == hipSuccess ? RL_OK : hip_fail(c, e, "rope launch");
        }
        case RL_K_GEMM_O:
            st = run_gemm_plan(c, kc, &p, c->ws + L.off_attn, HqD, lw(c->w.w_o, static_cast<size_t>(H) * HqD), M, H,
                               HqD, EPI_RESID, nullptr, 0, x, H, nullptr, 0, true, &splits);
            if (st != RL_OK) return st;
            return resid_then_norm(c, DT_BF16, splits, x, M, H, lw(c->w.mlp_norm, H), eps, h);
        case RL_K_GEMM_GATE_UP:
            return run_gemm_plan(c, kc, &p, h, H, lw(c->w.w_gate_up, static_cast<size_t>(2) * F * H), M, 2 * F, H,
                                 EPI_SWIGLU, nullptr, 0, nullptr, 0, c->ws + L.off_mlp, F, false, &splits);
        case RL_K_GEMM_DOWN:
            st = run_gemm_plan(c, kc, &p, c->ws + L.off_mlp, F, lw(c->w.w_down, static_cast<size_t>(H) * F), M, H, F,
                               EPI_RESID, nullptr, 0, x, H, nullptr, 0, true, &splits);
            if (st != RL_OK) return st;
            return resid_then_norm(c, DT_BF16, splits, x, M, H, lw(c->w.attn_norm, H), eps, h);
        default:
            return run_gemm_plan(c, kc, &p, h, H, c->w.lm_head, M, cf.vocab, H, EPI_F32, c->wsp<float>(L.off_logits),
                                 cf.vocab, nullptr, 0, nullptr, 0, false, &splits);
    }
}

struct TuneTimer {
    rl_decode_ctx* c;
    const int32_t* zeros;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    // mean microseconds per unit over `layers`, after one untimed unit on `warm`
    rl_status run(int kc, const GemmPlan& p, int M, const std::vector<int>& layers, int warm, float* us) {
        rl_status st = tune_unit(c, kc, p, M, warm, zeros);
        if (st != RL_OK) return st;
        hipError_t e = hipEventRecord(e0, c->stream);
        if (e != hipSuccess) return hip_fail(c, e, "event record");
        for (int l : layers) {
            st = tune_unit(c, kc, p, M, l, zeros);
            if (st != RL_OK) return st;
        }
        if ((e = hipEventRecord(e1, c->stream)) != hipSuccess) return hip_fail(c, e, "event record");
        if ((e = hipEventSynchronize(e1)) != hipSuccess) return hip_fail(c, e, "event synchronize");
        float ms = 0.0f;
        if ((e = hipEventElapsedTime(&ms, e0, e1)) != hipSuccess) return hip_fail(c, e, "event time");
        *us = ms * 1000.0f / static_cast<float>(layers.size());
        return RL_OK;
    }
};

constexpr int kTuneFinalists = 2;   // isolated-unit winners measured again inside decode steps
constexpr int kTuneCtx = 64;        // context of every row of a measuring step
constexpr int kTuneSteps = 2;       // timed measuring steps per finalist (after one untimed)

// Device time of a decode step of rows 0 .. M-1 at context ctx0 (mean over
// kTuneSteps steps after one untimed step).
struct TuneStepper {
    rl_decode_ctx* c;
    int32_t* tok = nullptr;   // device: zero input tokens, then output tokens and log-probs
    std::vector<int32_t> slots;
    std::vector<uint64_t> uids;
    int ctx0 = 0;
    rl_status time(int M, hipEvent_t e0, hipEvent_t e1, float* ms) {
        const rl_sample_params sp{0, 1.0f, 0};
        for (int i = 0; i < M; ++i) c->len[i] = ctx0;
        int32_t* out_tok = tok + c->cfg.max_seqs;
        float* out_lp = reinterpret_cast<float*>(tok + 2 * c->cfg.max_seqs);
        rl_status st = rl_decode_step(c, M, slots.data(), uids.data(), tok, nullptr, &sp, out_tok, out_lp, nullptr);
        if (st != RL_OK) return st;
        hipError_t e = hipEventRecord(e0, c->stream);
        if (e != hipSuccess) return hip_fail(c, e, "event record");
        for (int k = 0; k < kTuneSteps; ++k) {
            st = rl_decode_step(c, M, slots.data(), uids.data(), tok, nullptr, &sp, out_tok, out_lp, nullptr);
            if (st != RL_OK) return st;
        }
        if ((e = hipEventRecord(e1, c->stream)) != hipSuccess) return hip_fail(c, e, "event record");
        if ((e = hipEventSynchronize(e1)) != hipSuccess) return hip_fail(c, e, "event synchronize");
        if ((e = hipEventElapsedTime(ms, e0, e1)) != hipSuccess) return hip_fail(c, e, "event time");
        *ms /= kTuneSteps;
        return RL_OK;
    }
};

// For every batch size M (ascending) and decode GEMM class: every candidate
// plan is timed as an isolated unit over a few layers (consecutive
// candidates on disjoint layers, so that a layer's weights are not still
// cached from the previous candidate); then, one class at a time with the
// other classes at their current choice, the fastest few and the cost
// model's plan are each timed inside whole decode steps of M rows, which
// also price what a plan costs its neighbours, and the fastest step wins.
// The context holds no live sequence; the measuring steps use slots
// 0 .. M-1 at a short context and leave every length at 0.
rl_status tune_gemms(rl_decode_ctx* c, const std::vector<int>& sizes) {
    const rl_model_config& cf = c->cfg;
    const Layout& L = c->lay;
    const int H = cf.hidden, F = cf.ffn, HqD = cf.n_q_heads * cf.head_dim, NL = cf.n_layers;
    struct Shape { int kc, Nw, K, epi; };
    const Shape shapes[5] = {{RL_K_GEMM_QKV, L.nqkv, H, EPI_F32}, {RL_K_GEMM_O, H, HqD, EPI_RESID},
                             {RL_K_GEMM_GATE_UP, 2 * F, H, EPI_SWIGLU}, {RL_K_GEMM_DOWN, H, F, EPI_RESID},
                             {RL_K_GEMM_LM_HEAD, cf.vocab, H, EPI_F32}};
    const int order[5] = {2, 3, 0, 1, 4};   // step-level choice: largest share of the step first
    // finite operands: zero activations, positions, destinations and K/V
    // (no sequence is live, so the pool holds nothing to keep)
    hipError_t e = hipMemsetAsync(c->ws + L.off_x, 0, L.off_part - L.off_x, c->stream);
    if (e == hipSuccess) e = hipMemsetAsync(c->ws + L.off_tok, 0, static_cast<size_t>(L.R) * 4, c->stream);
    if (e == hipSuccess) e = hipMemsetAsync(c->kv, 0, L.kv_bytes, c->stream);
    if (e != hipSuccess) return hip_fail(c, e, "workspace clear");
    TuneTimer tm{c, c->wsp<int32_t>(L.off_tok)};
    TuneStepper stp{c};
    stp.ctx0 = std::max(0, std::min(kTuneCtx, cf.max_ctx - (kTuneSteps + 2)));
    const int max_m = sizes.back();
    for (int i = 0; i < max_m; ++i) {
        stp.slots.push_back(i);
        stp.uids.push_back(static_cast<uint64_t>(i));
    }
    if ((e = hipMalloc(&stp.tok, static_cast<size_t>(3) * cf.max_seqs * 4)) != hipSuccess)
        return hip_fail(c, e, "tuning buffers");
    e = hipMemsetAsync(stp.tok, 0, static_cast<size_t>(3) * cf.max_seqs * 4, c->stream);
    if (e == hipSuccess) e = hipEventCreate(&tm.e0);
    if (e == hipSuccess) e = hipEventCreate(&tm.e1);
    const uint32_t profile = c->profile;
    const rl_attn_plan_stats plan_stats = c->plan;
    c->profile = 0;
    rl_status st = e == hipSuccess ? RL_OK : hip_fail(c, e, "tuning set-up");
    std::vector<int> all(NL);
    for (int l = 0; l < NL; ++l) all[l] = l;
    std::vector<GemmPlan> cand[5];
    std::vector<float> unit_us[5];
    for (size_t si = 0; si < sizes.size() && st == RL_OK; ++si) {
        const int M = sizes[si];
        std::vector<int> fin[5];
        for (int k = 0; k < 5 && st == RL_OK; ++k) {
            const Shape& sh = shapes[k];
            const bool head = sh.kc == RL_K_GEMM_LM_HEAD;
            GemmPlan buf[kMaxGemmCandidates];
            const int n = plan_gemm_candidates(M, sh.Nw, sh.K, sh.epi, F, buf, kMaxGemmCandidates);
            cand[k].assign(buf, buf + n);
            unit_us[k].assign(n, 0.0f);
            std::vector<std::pair<float, int>> first;
            for (int i = 0; i < n && st == RL_OK; ++i) {
                std::vector<int> lay;
                int warm = 0;
                if (head) {
                    lay = {0};
                } else if (NL < 5) {
                    lay = all;
                } else {
                    warm = (5 * i) % NL;
                    for (int q = 1; q <= 4; ++q) lay.push_back((warm + q) % NL);
                }
                st = tm.run(sh.kc, cand[k][i], M, lay, warm, &unit_us[k][i]);
                first.emplace_back(unit_us[k][i], i);
            }
            std::sort(first.begin(), first.end());
            fin[k].push_back(0);   // the cost model's plan
            for (int j = 0; j < static_cast<int>(first.size()) && static_cast<int>(fin[k].size()) <= kTuneFinalists; ++j)
                if (first[j].second != 0) fin[k].push_back(first[j].second);
        }
        if (st != RL_OK) break;
        // this size's entries, at the cost model's plans; sizes ascend, so a
        // lookup at M finds these before any larger size's
        const size_t base = c->tuned.size();
        for (int k = 0; k < 5; ++k)
            c->tuned.push_back({shapes[k].kc, M, shapes[k].Nw, shapes[k].K, shapes[k].epi, cand[k][0], unit_us[k][0]});
        for (int oi = 0; oi < 5 && st == RL_OK; ++oi) {
            const int k = order[oi];
            if (fin[k].size() < 2) continue;
            int best = -1;
            float best_ms = 0.0f;
            for (int i : fin[k]) {
                c->tuned[base + k].p = cand[k][i];
                float ms = 0.0f;
                st = stp.time(M, tm.e0, tm.e1, &ms);
                if (st != RL_OK) break;
                if (best < 0 || ms < best_ms) { best = i; best_ms = ms; }
            }
            if (st != RL_OK) break;
            c->tuned[base + k].p = cand[k][best];
            c->tuned[base + k].us = unit_us[k][best];
        }
    }
    std::vector<std::pair<int, int>> none;
    for (int i = 0; i < max_m; ++i) {
        c->len[i] = 0;
        none.emplace_back(i, 0);
    }
    set_pages(c, none);
    c->profile = profile;
    c->plan = plan_stats;
    if (tm.e0) (void)hipEventDestroy(tm.e0);
    if (tm.e1) (void)hipEventDestroy(tm.e1);
    (void)hipStreamSynchronize(c->stream);
    (void)hipFree(stp.tok);
    if (st != RL_OK) {
        c->tuned.clear();
        return st;
    }
    std::stable_sort(c->tuned.begin(), c->tuned.end(),
                     [](const rl_decode_ctx::TunedPlan& a, const rl_decode_ctx::TunedPlan& b) {
                         return a.kc != b.kc ? a.kc < b.kc : a.M < b.M;
                     });
    return RL_OK;
}

// Split-KV work items for a set of query blocks.  Each block: nq tokens at
// positions pos0 .. pos0+nq-1 of a slot, keys [0, pos0 + nq).  With src >= 0
// the keys [0, plen) (plen a multiple of 32, <= pos0) are read from slot src
// instead (a shared prompt) and the rest from the block's own slot.
struct Block {
    int qrow, nq, slot, pos0;
    int src = -1, plen = 0;
};

int block_items(const Block& b, int C) {
    const int hi = b.pos0 + b.nq;
    if (b.src >= 0 && b.plen > 0) return ceil_div(b.plen, C) + ceil_div(hi - b.plen, C);
    return ceil_div(hi, C);
}

int choose_chunk(const std::vector<Block>& blocks, int Hkv, int64_t forced, int default_min,
                 int items_cap, bool decode) {
    auto count = [&](int C, long* items, long* multi, int* most) {
        *items = 0; *multi = 0; *most = 0;
        for (const Block& b : blocks) {
            const long k = block_items(b, C);
            *items += k;
            if (k > 1) *multi += k;
            *most = std::max<int>(*most, static_cast<int>(k));
        }
    };
    long items, multi;
    int most, C;
    if (forced > 0) {
        C = static_cast<int>(forced);
    } else if (decode) {
        bool shared = false;
        for (const Block& b : blocks) shared = shared || (b.src >= 0 && b.plen > 0);
        if (shared) {
            // Prompt chunks served from L2 and HBM-bound own parts take very
            // different times per key: short items let the dispatcher balance
            // them over the chip.  Over a GRPO rollout, 256 keys per item took
            // 7.4% less attention time than the long-item rule (512: 6.8% less,
            // 128: 1% less).
            C = kSharedDecodeChunk;
            // few rows: shorter items, so that enough waves stream the keys
            while (C > 64) {
                count(C, &items, &multi, &most);
                if (items * Hkv >= 2 * kAttnWaveTarget) break;
                C /= 2;
            }
        } else {
            C = 64;
            while (C < (1 << 16)) {
                count(2 * C, &items, &multi, &most);
                if (items * Hkv < kAttnWaveTarget) break;
                C *= 2;
            }
        }
    } else {
        C = default_min;
    }
    for (;;) {
        count(C, &items, &multi, &most);
        const bool fits = items <= items_cap && multi <= kPartItems && most <= kMaxCombine;
        if (fits || C >= (1 << 20)) break;
        C *= 2;
    }
    return C;
}

// Work-item order for shared prompts.  The attention grid is (items / 4,
// Hkv) with the x extent a multiple of 8, so workgroup x runs on XCD x % 8
// for every kv-head, and workgroups start in x order.  Items that read the
// same shared chunk (the prompt of one group) are kept together and their
// workgroups placed on one XCD, so the chunk comes from HBM once and the
// other reads hit that XCD's L2.  Workgroups (4 consecutive items; a run of
// up to kMaxRunUnits of them for one chunk stays whole) are dealt longest first to the XCD with
// the least work, so each XCD also starts its longest ones first.  Returns
// the item order (new position -> old index, -1 = empty padding item).
constexpr int kMaxRunUnits = 4;   // a chunk read by more workgroups spreads over several XCDs

std::vector<int> place_shared(const std::vector<AttnItem>& its, const std::vector<int64_t>& key) {
    std::vector<int> idx(its.size());
    for (size_t i = 0; i < idx.size(); ++i) idx[i] = static_cast<int>(i);
    std::stable_sort(idx.begin(), idx.end(), [&](int a, int b) {
        const bool sa = key[a] >= 0, sb = key[b] >= 0;
        if (sa != sb) return sa;
        return sa && key[a] < key[b];
    });
    const int nu = static_cast<int>((idx.size() + 3) / 4);
    // unit time: its longest item; runs: consecutive units of one chunk
    std::vector<int> utime(nu, 0);
    struct Run { int u0, u1, t; };
    std::vector<Run> runs;
    for (int u = 0; u < nu; ++u) {
        const int b0 = 4 * u, b1 = std::min<int>(4 * u + 4, static_cast<int>(idx.size()));
        for (int i = b0; i < b1; ++i) utime[u] = std::max(utime[u], its[idx[i]].kv_hi - its[idx[i]].kv_lo);
        const int64_t k = key[idx[b0]];
        if (u > 0 && k >= 0 && k == key[idx[4 * u - 1]] && runs.back().u1 - runs.back().u0 < kMaxRunUnits) {
            runs.back().u1 = u + 1;
            runs.back().t = std::max(runs.back().t, utime[u]);
        } else {
            runs.push_back(Run{u, u + 1, utime[u]});
        }
    }
    std::stable_sort(runs.begin(), runs.end(), [](const Run& a, const Run& b) { return a.t > b.t; });
    std::vector<std::vector<int>> q(8);
    double load[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (const Run& r : runs) {
        int qq = 0;
        for (int j = 1; j < 8; ++j) if (load[j] < load[qq]) qq = j;
        for (int u = r.u0; u < r.u1; ++u) {
            q[qq].push_back(u);
            load[qq] += utime[u];
        }
    }
    size_t L = 0;
    for (int j = 0; j < 8; ++j) L = std::max(L, q[j].size());
    std::vector<int> order(32 * L, -1);
    for (int j = 0; j < 8; ++j)
        for (size_t i = 0; i < q[j].size(); ++i) {
            const int u = q[j][i];
            const size_t x = 8 * i + j;
            for (int t = 0; t < 4 && 4 * u + t < static_cast<int>(idx.size()); ++t) order[4 * x + t] = idx[4 * u + t];
        }
    return order;
}

rl_status build_items(rl_decode_ctx* c, Meta* m, const std::vector<Block>& blocks, int C, Fwd* f) {
    std::vector<AttnItem> its;
    std::vector<int64_t> key;
    std::vector<int> split_first;
    int part = 0;
    bool any_shared = false;
    double scorepos = 0, kvpos = 0;
    for (const Block& b : blocks) {
        const int hi_all = b.pos0 + b.nq;
        const bool sh = b.src >= 0 && b.plen > 0;
        const int n_sh = sh ? ceil_div(b.plen, C) : 0;
        const int lo_own = sh ? b.plen : 0;
        const int nch = n_sh + ceil_div(hi_all - lo_own, C);
        const int part0 = nch > 1 ? part : -1;
        if (nch > kMaxCombine) return fail(c, RL_ERR_CAPACITY, "too many split-KV chunks in one block");
        // the combine reads the block's rows and partial range from its last
        // item (an own-slot item: never merged into a pair)
        if (nch > 1) split_first.push_back(static_cast<int>(its.size()) + nch - 1);
        for (int ch = 0; ch < nch; ++ch) {
            AttnItem it;
            std::memset(&it, 0, sizeof(it));
            it.qrow = b.qrow; it.nq = b.nq; it.pos0 = b.pos0;
            it.qrow_b = -1; it.part_b = -1;
            if (ch < n_sh) {
                it.slot = b.src;
                it.kv_lo = ch * C;
                it.kv_hi = std::min(b.plen, (ch + 1) * C);
                key.push_back((static_cast<int64_t>(b.src) << 32) | ch);
                any_shared = true;
            } else {
                const int j = ch - n_sh;
                it.slot = b.slot;
                it.kv_lo = lo_own + j * C;
                it.kv_hi = std::min(hi_all, lo_own + (j + 1) * C);
                key.push_back(-1);
            }
            it.part = nch > 1 ? part++ : -1;
            it.part0 = part0;
            it.nparts = nch;
            its.push_back(it);
        }
        for (int t = 0; t < b.nq; ++t) scorepos += b.pos0 + t + 1;
        kvpos += sh ? hi_all - b.plen : hi_all;
    }
    if (part > kPartItems) return fail(c, RL_ERR_CAPACITY, "too many split-KV partials");
    std::vector<int> order;
    const int G = c->cfg.n_q_heads / c->cfg.n_kv_heads;
    if (any_shared && 2 * G <= 16) {
        // single-token readers of one shared chunk go two to an item
        std::vector<int> sidx;
        for (size_t i = 0; i < its.size(); ++i)
            if (key[i] >= 0 && its[i].nq == 1) sidx.push_back(static_cast<int>(i));
        std::stable_sort(sidx.begin(), sidx.end(), [&](int a, int b) { return key[a] < key[b]; });
        std::vector<char> drop(its.size(), 0);
        for (size_t k = 0; k + 1 < sidx.size();) {
            const int a = sidx[k], b = sidx[k + 1];
            if (key[a] != key[b]) { ++k; continue; }
            its[a].nq = 2;
            its[a].qrow_b = its[b].qrow;
            its[a].part_b = its[b].part;
            drop[b] = 1;
            k += 2;
        }
        std::vector<int> remap(its.size(), -1);
        size_t w = 0;
        for (size_t i = 0; i < its.size(); ++i) {
            if (drop[i]) continue;
            remap[i] = static_cast<int>(w);
            its[w] = its[i];
            key[w] = key[i];
            ++w;
        }
        for (int& f0 : split_first) f0 = remap[f0];
        its.resize(w);
        key.resize(w);
    }
    if (any_shared) {
        order = place_shared(its, key);
        if (order.size() > static_cast<size_t>(c->lay.items_cap)) order.clear();   // keep the plain order
        // algorithmic KV positions: the own parts plus each shared chunk once
        std::vector<std::pair<int64_t, int>> sh;
        for (size_t i = 0; i < its.size(); ++i)
            if (key[i] >= 0) sh.emplace_back(key[i], its[i].kv_hi - its[i].kv_lo);
        std::sort(sh.begin(), sh.end());
        for (size_t i = 0; i < sh.size(); ++i)
            if (i == 0 || sh[i].first != sh[i - 1].first) kvpos += sh[i].second;
        f->attn_kv_positions = kvpos;
    }
    if (order.empty()) {
        order.resize(its.size());
        for (size_t i = 0; i < its.size(); ++i) order[i] = static_cast<int>(i);
    }
    if (order.size() > static_cast<size_t>(c->lay.items_cap)) return fail(c, RL_ERR_CAPACITY, "too many attention work items");
    AttnItem* dItems = nullptr;
    AttnItem* items = m->take<AttnItem>(order.size(), &dItems);
    int32_t* dSplit = nullptr;
    int32_t* split = m->take<int32_t>(std::max<size_t>(split_first.size(), 1), &dSplit);
    if (!items || !split) return fail(c, RL_ERR_CAPACITY, "per-call metadata exceeds its workspace region");
    std::vector<int> newpos(its.size(), 0);
    for (size_t x = 0; x < order.size(); ++x) {
        if (order[x] < 0) {   // padding: no query columns, no keys
            std::memset(&items[x], 0, sizeof(AttnItem));
            items[x].part = -1;
            items[x].qrow_b = -1;
            items[x].part_b = -1;
        } else {
            items[x] = its[order[x]];
            newpos[order[x]] = static_cast<int>(x);
        }
    }
    for (size_t i = 0; i < split_first.size(); ++i) split[i] = newpos[split_first[i]];
    f->plan_items = f->plan_shared = f->plan_pairs = f->plan_lds = 0;
    for (size_t x = 0; x < order.size(); ++x) {
        if (order[x] < 0) continue;
        f->plan_items += 1;
        f->plan_shared += key[order[x]] >= 0;
        f->plan_pairs += its[order[x]].qrow_b >= 0;
    }
    if (any_shared) {   // workgroups whose four items read one shared chunk stage it through LDS
        for (size_t x = 0; x + 3 < order.size(); x += 4) {
            bool same = order[x] >= 0 && key[order[x]] >= 0;
            for (int t = 1; t < 4 && same; ++t) same = order[x + t] >= 0 && key[order[x + t]] == key[order[x]];
            if (same) {
                items[x].pad = 1;
                f->plan_lds += 1;
            }
        }
    }
    f->items = dItems;
    f->n_items = static_cast<int>(order.size());
    f->n_partial_items = part;
    f->split_blocks = dSplit;
    f->n_split_blocks = static_cast<int>(split_first.size());
    f->attn_score_positions = scorepos;
    return RL_OK;
}

// Prefill / scoring tiles: each block run of consecutive query tokens of one
// sequence (blocks of one slot with consecutive rows and positions) split
// into tiles of kPrefillWaves * (16 / G) tokens, longest key range first.
rl_status build_tiles(rl_decode_ctx* c, Meta* m, const std::vector<Block>& blocks, Fwd* f) {
    const int G = c->cfg.n_q_heads / c->cfg.n_kv_heads;
    const int T = kPrefillWaves * std::max(1, 16 / G);
    std::vector<PrefillTile> tl;
    size_t i = 0;
    while (i < blocks.size()) {
        // a run: consecutive blocks continuing the same sequence segment
        size_t j = i + 1;
        while (j < blocks.size() && blocks[j].slot == blocks[i].slot &&
               blocks[j].qrow == blocks[j - 1].qrow + blocks[j - 1].nq &&
               blocks[j].pos0 == blocks[j - 1].pos0 + blocks[j - 1].nq)
            ++j;
        const int qrow0 = blocks[i].qrow, pos0 = blocks[i].pos0, slot = blocks[i].slot;
        const int n = blocks[j - 1].qrow + blocks[j - 1].nq - qrow0;
        for (int t = 0; t < n; t += T) tl.push_back(PrefillTile{qrow0 + t, std::min(T, n - t), slot, pos0 + t});
        i = j;
    }
    std::stable_sort(tl.begin(), tl.end(), [](const PrefillTile& a, const PrefillTile& b) {
        return a.pos0 + a.ntok > b.pos0 + b.ntok;
    });
    PrefillTile* d = nullptr;
    PrefillTile* h = m->take<PrefillTile>(std::max<size_t>(tl.size(), 1), &d);
    if (!h) return fail(c, RL_ERR_CAPACITY, "per-call metadata exceeds its workspace region");
    std::copy(tl.begin(), tl.end(), h);
    double scorepos = 0;
    for (const Block& b : blocks)
        for (int t = 0; t < b.nq; ++t) scorepos += b.pos0 + t + 1;
    f->tiles = d;
    f->n_tiles = static_cast<int>(tl.size());
    f->n_items = 0;
    f->n_split_blocks = 0;
    f->attn_score_positions = scorepos;
    return RL_OK;
}

// Drop prompt sharing of the given slots, and of every slot that reads its
// prompt from one of them (their own copies stay valid).
void unshare(rl_decode_ctx* c, int n, const int32_t* slots) {
    const int S = c->cfg.max_seqs;
    std::vector<char> hit(static_cast<size_t>(S), 0);
    for (int i = 0; i < n; ++i) hit[slots[i]] = 1;
    for (int s = 0; s < S; ++s)
        if (hit[s] || (c->share_src[s] >= 0 && hit[c->share_src[s]])) {
            c->share_src[s] = -1;
            c->share_len[s] = 0;
        }
}

void fill_rope_table(const rl_model_config& c, int cap, std::vector<float>* out) {
    const int half = c.head_dim / 2;
    out->assign(static_cast<size_t>(cap) * half * 2, 0.0f);
    for (int i = 0; i < half; ++i) {
        const double w = std::pow(c.rope_theta, -2.0 * i / static_cast<double>(c.head_dim));
        for (int p = 0; p < cap; ++p) {
            const double a = static_cast<double>(p) * w;
            (*out)[static_cast<size_t>(p) * half + i] = static_cast<float>(std::cos(a));
            (*out)[static_cast<size_t>(cap) * half + static_cast<size_t>(p) * half + i] = static_cast<float>(std::sin(a));
        }
    }
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

rl_status check_sp(rl_decode_ctx* c, const rl_sample_params* sp) {
    if (!sp) return fail(c, RL_ERR_INVALID_ARG, "sample params are NULL");
    if (sp->reserved != 0) return fail(c, RL_ERR_INVALID_ARG, "sample_params.reserved must be 0");
    if (!(sp->temperature >= 0.0f) || !std::isfinite(sp->temperature))
        return fail(c, RL_ERR_INVALID_ARG, "temperature must be finite and >= 0");
    return RL_OK;
}

rl_status check_slots(rl_decode_ctx* c, int n, const int32_t* slots, std::vector<char>* seen) {
    seen->assign(static_cast<size_t>(c->cfg.max_seqs), 0);
    for (int i = 0; i < n; ++i) {
        const int s = slots[i];
        if (s < 0 || s >= c->cfg.max_seqs) return fail(c, RL_ERR_INVALID_ARG, "slot out of range");
        if ((*seen)[s]) return fail(c, RL_ERR_INVALID_ARG, "duplicate slot");
        (*seen)[s] = 1;
    }
    return RL_OK;
}

struct DeviceGuard {
    int prev = -1;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev) == hipSuccess && prev != dev) (void)hipSetDevice(dev);
        else prev = -1;
    }
    ~DeviceGuard() { if (prev >= 0) (void)hipSetDevice(prev); }
};

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================
extern "C" {

const char* rl_status_string(rl_status s) {
    switch (s) {
        case RL_OK: return "ok";
        case RL_ERR_INVALID_ARG: return "invalid argument";
        case RL_ERR_UNSUPPORTED: return "unsupported shape";
        case RL_ERR_CAPACITY: return "capacity exceeded";
        case RL_ERR_HIP: return "HIP runtime error";
        case RL_ERR_STATE: return "invalid or destroyed context";
    }
    return "unknown status";
}

const char* rl_decode_last_error(const rl_decode_ctx* ctx) {
    if (!ctx_ok(ctx)) return "invalid or destroyed context";
    return ctx->err.c_str();
}

size_t rl_decode_kv_bytes(const rl_model_config* cfg) {
    rl_status s; std::string why;
    if (!cfg_check(cfg, &s, &why)) return 0;
    return make_layout(*cfg).kv_bytes;
}

size_t rl_decode_workspace_bytes(const rl_model_config* cfg) {
    rl_status s; std::string why;
    if (!cfg_check(cfg, &s, &why)) return 0;
    return make_layout(*cfg).ws_bytes;
}

namespace {

// RoPE table in the workspace; synchronises the stream.
hipError_t init_workspace(rl_decode_ctx* c) {
    std::vector<float> table;
    fill_rope_table(c->cfg, c->lay.cap, &table);
    hipError_t e = hipMemcpyAsync(c->ws + c->lay.off_rope, table.data(), table.size() * sizeof(float),
                                  hipMemcpyHostToDevice, c->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
    return e;
}

// Every weight the model reads is given and 16-byte aligned (a mixture of
// experts reads the router and experts instead of w_gate_up / w_down).
bool weights_ok(const rl_model_config& c, const rl_weights* w) {
    if (!w) return false;
    const bool moe = c.n_experts > 0;
    const void* wp[10] = {w->embed, w->attn_norm, w->w_qkv, w->w_o, w->mlp_norm, w->final_norm, w->lm_head,
                          moe ? w->w_router : w->w_gate_up, moe ? w->w_exp_gate_up : w->w_down,
                          moe ? w->w_exp_down : w->w_down};
    for (const void* p : wp)
        if (!p || !aligned(p, 16)) return false;
    return true;
}

}  // namespace

rl_status rl_decode_create(const rl_model_config* cfg, const rl_weights* w, void* kv_pool,
                           size_t kv_bytes, void* workspace, size_t ws_bytes, void* stream,
                           rl_decode_ctx** out) {
    if (!out) return RL_ERR_INVALID_ARG;
    *out = nullptr;
    rl_status code; std::string why;
    if (!cfg_check(cfg, &code, &why)) return code;
    if (!weights_ok(*cfg, w)) return RL_ERR_INVALID_ARG;
    if (!kv_pool || !workspace || !aligned(kv_pool, 256) || !aligned(workspace, 256)) return RL_ERR_INVALID_ARG;
    Layout L = make_layout(*cfg);
    if (kv_bytes < L.kv_bytes || ws_bytes < L.ws_bytes) return RL_ERR_CAPACITY;

    rl_decode_ctx* c = new (std::nothrow) rl_decode_ctx();
    if (!c) return RL_ERR_CAPACITY;
    c->cfg = *cfg;
    c->w = *w;
    c->lay = L;
    c->kv = static_cast<uint8_t*>(kv_pool);
    c->ws = static_cast<uint8_t*>(workspace);
    c->stream = static_cast<hipStream_t>(stream);
    c->len.assign(static_cast<size_t>(cfg->max_seqs), 0);
    c->share_src.assign(static_cast<size_t>(cfg->max_seqs), -1);
    c->share_len.assign(static_cast<size_t>(cfg->max_seqs), 0);
    if (c->paged()) {
        c->ptab.assign(static_cast<size_t>(cfg->max_seqs) * L.maxp, -1);
        c->npages.assign(static_cast<size_t>(cfg->max_seqs), 0);
        c->free_pages.resize(static_cast<size_t>(L.pages));
        for (int i = 0; i < L.pages; ++i) c->free_pages[i] = L.pages - 1 - i;   // handed out from page 0 up
        c->pref.assign(static_cast<size_t>(L.pages), 0);
    }
    auto cleanup = [&](rl_status s) {
        for (int i = 0; i < kStages; ++i) {
            if (c->staging[i]) (void)hipHostFree(c->staging[i]);
            if (c->stage_ev[i]) (void)hipEventDestroy(c->stage_ev[i]);
        }
        delete c;
        return s;
    };
    if (hipGetDevice(&c->device) != hipSuccess) return cleanup(RL_ERR_HIP);
    for (int i = 0; i < kStages; ++i) {
        if (hipHostMalloc(reinterpret_cast<void**>(&c->staging[i]), L.meta_bytes, hipHostMallocDefault) != hipSuccess)
            return cleanup(RL_ERR_HIP);
        if (hipEventCreateWithFlags(&c->stage_ev[i], hipEventDisableTiming) != hipSuccess)
            return cleanup(RL_ERR_HIP);
    }
    if (init_workspace(c) != hipSuccess) return cleanup(RL_ERR_HIP);
    for (int i = 0; i < RL_K_COUNT; ++i)
        std::snprintf(c->stats[i].name, sizeof(c->stats[i].name), "%s", kClassNames[i]);
    *out = c;
    return RL_OK;
}

rl_status rl_decode_destroy(rl_decode_ctx* ctx) {
    if (!ctx) return RL_OK;
    if (!ctx_ok(ctx)) return RL_ERR_STATE;
    DeviceGuard g(ctx->device);
    (void)hipStreamSynchronize(ctx->stream);
    for (auto& p : ctx->pending) { (void)hipEventDestroy(p.a); (void)hipEventDestroy(p.b); }
    for (hipEvent_t e : ctx->ev_pool) (void)hipEventDestroy(e);
    for (int i = 0; i < kStages; ++i) {
        if (ctx->staging[i]) (void)hipHostFree(ctx->staging[i]);
        if (ctx->stage_ev[i]) (void)hipEventDestroy(ctx->stage_ev[i]);
    }
    ctx->magic = kDead;
    delete ctx;
    return RL_OK;
}

rl_status rl_prefill(rl_decode_ctx* ctx, int32_t n_prompts, int32_t group, const int32_t* slots,
                     const uint64_t* seq_uids, const int32_t* prompt_offsets, const int32_t* tokens,
                     const void* embeds, int32_t n_embed_rows, const int32_t* forced_first,
                     const rl_sample_params* sp, int32_t* out_tok, float* out_logp, float* out_logits) {
    if (!ctx_ok(ctx)) return RL_ERR_STATE;
    rl_decode_ctx* c = ctx;
    const rl_model_config& cf = c->cfg;
    if (n_prompts < 1 || group < 1) return fail(c, RL_ERR_INVALID_ARG, "n_prompts and group must be >= 1");
    if (static_cast<int64_t>(n_prompts) * group > cf.max_seqs)
        return fail(c, RL_ERR_CAPACITY, "n_prompts * group exceeds max_seqs");
    if (!slots || !seq_uids || !prompt_offsets || !tokens || !out_tok || !out_logp)
        return fail(c, RL_ERR_INVALID_ARG, "required pointer is NULL");
    if (n_embed_rows < 0 || (n_embed_rows > 0 && !embeds)) return fail(c, RL_ERR_INVALID_ARG, "bad embedding rows");
    if (embeds && !aligned(embeds, 16)) return fail(c, RL_ERR_INVALID_ARG, "embeds must be 16-byte aligned");
    if (out_logits && !aligned(out_logits, 16)) return fail(c, RL_ERR_INVALID_ARG, "out_logits must be 16-byte aligned");
    rl_status st = check_sp(c, sp);
    if (st != RL_OK) return st;
    const int n_out = n_prompts * group;
    std::vector<char> seen;
    st = check_slots(c, n_out, slots, &seen);
    if (st != RL_OK) return st;
    if (prompt_offsets[0] != 0) return fail(c, RL_ERR_INVALID_ARG, "prompt_offsets[0] must be 0");
    int64_t total = 0;
    for (int p = 0; p < n_prompts; ++p) {
        const int64_t len = static_cast<int64_t>(prompt_offsets[p + 1]) - prompt_offsets[p];
        if (len < 1) return fail(c, RL_ERR_INVALID_ARG, "empty prompt");
        if (len > cf.max_ctx - 1) return fail(c, RL_ERR_CAPACITY, "prompt longer than max_ctx - 1");
        total += len;
    }
    if (total > cf.max_prefill_tokens) return fail(c, RL_ERR_CAPACITY, "prompts exceed max_prefill_tokens");
    const int R = static_cast<int>(total);
    std::vector<int> plens(static_cast<size_t>(n_prompts));
    for (int p = 0; p < n_prompts; ++p) plens[p] = prompt_offsets[p + 1] - prompt_offsets[p];
    std::vector<int32_t> new_len(static_cast<size_t>(n_out));
    for (int o = 0; o < n_out; ++o) new_len[o] = plens[o / group];
    if (!group_pages_fit(c, n_prompts, group, slots, plens, new_len))
        return fail(c, RL_ERR_CAPACITY, "not enough free K/V pages");
    DeviceGuard g(c->device);

    Meta m{};
    int stage = 0;
    st = begin_meta(c, &m, &stage);
    if (st != RL_OK) return st;
    const PageStage ps = take_pages(c, &m);
    int32_t *d_row_pos, *d_row_dst, *d_row_slot, *d_dst, *d_lrow, *d_posn, *d_last;
    uint64_t* d_uid;
    int32_t* row_pos = m.take<int32_t>(R, &d_row_pos);
    int32_t* row_dst = m.take<int32_t>(R, &d_row_dst);
    int32_t* row_slot = m.take<int32_t>(R, &d_row_slot);
    int32_t* dst = m.take<int32_t>(n_out, &d_dst);
    int32_t* lrow = m.take<int32_t>(n_out, &d_lrow);
    int32_t* posn = m.take<int32_t>(n_out, &d_posn);
    int32_t* last = m.take<int32_t>(n_prompts, &d_last);
    uint64_t* uid = m.take<uint64_t>(n_out, &d_uid);
    if (m.overflow) return fail(c, RL_ERR_CAPACITY, "per-call metadata exceeds its workspace region");
    std::vector<Block> blocks;
    const int G = cf.n_q_heads / cf.n_kv_heads;
    const int tq = std::max(1, 16 / G);
    double kvpos = 0;
    for (int p = 0; p < n_prompts; ++p) {
        const int b = prompt_offsets[p], len = prompt_offsets[p + 1] - b;
        // rows in the group's shared pages are written once, through its first slot
        const int shared_rows = shared_prompt_pages(c, len) * c->lay.page;
        for (int t = 0; t < len; ++t) {
            row_pos[b + t] = t;
            row_dst[b + t] = t < shared_rows ? -(slots[p * group] + 1) : p * group;
            row_slot[b + t] = slots[p * group];
        }
        last[p] = b + len - 1;
        for (int k = 0; k < group; ++k) {
            const int o = p * group + k;
            dst[o] = slots[o];
            lrow[o] = p;
            posn[o] = len;
            uid[o] = seq_uids[o];
        }
        for (int t = 0; t < len; t += tq) blocks.push_back(Block{b + t, std::min(tq, len - t), slots[p * group], t});
        kvpos += len;
    }
    Fwd f;
    f.rows = R;
    f.tok = tokens;
    f.embeds = embeds;
    f.n_embed_rows = n_embed_rows;
    f.row_pos = d_row_pos;
    f.row_dst = d_row_dst;
    f.n_dst = group;
    f.dst_slots = d_dst;
    f.row_slot = d_row_slot;
    f.attn_kv_positions = kvpos;
    if (c->bf16() && c->opt_prefill_items) {
        const int C = choose_chunk(blocks, cf.n_kv_heads, c->opt_chunk, kPrefillChunk, c->lay.items_cap, false);
        st = build_items(c, &m, blocks, C, &f);
        if (st != RL_OK) return st;
    } else if (c->bf16()) {
        st = build_tiles(c, &m, blocks, &f);
        if (st != RL_OK) return st;
    } else {
        double sp_ = 0;
        for (int p = 0; p < n_prompts; ++p) {
            const double len = prompt_offsets[p + 1] - prompt_offsets[p];
            sp_ += len * (len + 1) / 2;
        }
        f.attn_score_positions = sp_;
    }
    f.final_sel = d_last;
    f.n_final = n_prompts;
    f.logits = out_logits ? out_logits : c->wsp<float>(c->lay.off_logits);
    f.n_out = n_out;
    f.logit_row = d_lrow;
    f.uid = d_uid;
    f.pos_new = d_posn;
    f.forced = forced_first;
    f.seed = sp->seed;
    f.T = sp->temperature;
    f.out_tok = out_tok;
    f.out_logp = out_logp;
    set_group_pages(c, n_prompts, group, slots, plens, new_len);
    f.kvp = fill_pages(c, ps);
    st = upload_meta(c, &m, stage);
    if (st != RL_OK) return st;
    st = run_forward(c, f);
    if (st != RL_OK) return st;
    unshare(c, n_out, slots);
    for (int p = 0; p < n_prompts; ++p) {
        const int len = prompt_offsets[p + 1] - prompt_offsets[p];
        for (int k = 0; k < group; ++k) {
            const int s = slots[p * group + k];
            c->len[s] = len;
            if (group > 1) {   // every slot of the group holds the same prompt K/V
                c->share_src[s] = slots[p * group];
                c->share_len[s] = len;
            }
        }
    }
    return RL_OK;
}

rl_status rl_score(rl_decode_ctx* ctx, int32_t n_prompts, int32_t group, const int32_t* slots,
                   const int32_t* prompt_offsets, const int32_t* prompt_tokens, const void* embeds,
                   int32_t n_embed_rows, const int32_t* resp_offsets, const int32_t* resp_tokens,
                   float temperature, float* out_logp) {
    if (!ctx_ok(ctx)) return RL_ERR_STATE;
    rl_decode_ctx* c = ctx;
    const rl_model_config& cf = c->cfg;
    if (n_prompts < 1 || group < 1) return fail(c, RL_ERR_INVALID_ARG, "n_prompts and group must be >= 1");
    if (static_cast<int64_t>(n_prompts) * group > cf.max_seqs)
        return fail(c, RL_ERR_CAPACITY, "n_prompts * group exceeds max_seqs");
    if (!slots || !prompt_offsets || !prompt_tokens || !resp_offsets || !resp_tokens || !out_logp)
        return fail(c, RL_ERR_INVALID_ARG, "required pointer is NULL");
    if (n_embed_rows < 0 || (n_embed_rows > 0 && !embeds)) return fail(c, RL_ERR_INVALID_ARG, "bad embedding rows");
    if (embeds && !aligned(embeds, 16)) return fail(c, RL_ERR_INVALID_ARG, "embeds must be 16-byte aligned");
    if (!(temperature >= 0.0f) || !std::isfinite(temperature))
        return fail(c, RL_ERR_INVALID_ARG, "temperature must be finite and >= 0");
    const int n_seq = n_prompts * group;
    std::vector<char> seen;
    rl_status st = check_slots(c, n_seq, slots, &seen);
    if (st != RL_OK) return st;
    if (prompt_offsets[0] != 0) return fail(c, RL_ERR_INVALID_ARG, "prompt_offsets[0] must be 0");
    if (resp_offsets[0] != 0) return fail(c, RL_ERR_INVALID_ARG, "resp_offsets[0] must be 0");
    int64_t r1 = 0, r2 = 0;
    for (int p = 0; p < n_prompts; ++p) {
        const int64_t len = static_cast<int64_t>(prompt_offsets[p + 1]) - prompt_offsets[p];
        if (len < 1) return fail(c, RL_ERR_INVALID_ARG, "empty prompt");
        if (len > cf.max_ctx - 1) return fail(c, RL_ERR_CAPACITY, "prompt longer than max_ctx - 1");
        r1 += len;
        for (int k = 0; k < group; ++k) {
            const int sq = p * group + k;
            const int64_t m = static_cast<int64_t>(resp_offsets[sq + 1]) - resp_offsets[sq];
            if (m < 1) return fail(c, RL_ERR_INVALID_ARG, "empty response");
            if (len + m > cf.max_ctx) return fail(c, RL_ERR_CAPACITY, "prompt + response longer than max_ctx");
            r2 += m;
        }
    }
    if (r1 + r2 > cf.max_prefill_tokens)
        return fail(c, RL_ERR_CAPACITY, "prompt + response tokens exceed max_prefill_tokens");
    const int R1 = static_cast<int>(r1), R = static_cast<int>(r1 + r2);
    const int n_sel = n_prompts + static_cast<int>(r2) - n_seq;   // LM-head rows
    // each slot holds its group's prompt and its own response while scoring
    std::vector<int> plens(static_cast<size_t>(n_prompts));
    for (int p = 0; p < n_prompts; ++p) plens[p] = prompt_offsets[p + 1] - prompt_offsets[p];
    std::vector<int32_t> new_len(static_cast<size_t>(n_seq));
    for (int sq = 0; sq < n_seq; ++sq) new_len[sq] = plens[sq / group] + resp_offsets[sq + 1] - resp_offsets[sq];
    if (!group_pages_fit(c, n_prompts, group, slots, plens, new_len))
        return fail(c, RL_ERR_CAPACITY, "not enough free K/V pages");
    DeviceGuard g(c->device);

    Meta m{};
    int stage = 0;
    st = begin_meta(c, &m, &stage);
    if (st != RL_OK) return st;
    const PageStage ps = take_pages(c, &m);
    int32_t *d_row_pos, *d_row_dst, *d_row_slot, *d_dst, *d_sel, *d_items, *d_idx;
    int32_t* row_pos = m.take<int32_t>(R, &d_row_pos);
    int32_t* row_dst = m.take<int32_t>(R, &d_row_dst);
    int32_t* row_slot = m.take<int32_t>(R, &d_row_slot);
    int32_t* dst = m.take<int32_t>(n_seq, &d_dst);
    int32_t* sel = m.take<int32_t>(n_sel, &d_sel);
    int32_t* items = m.take<int32_t>(static_cast<size_t>(n_sel) + 1, &d_items);
    int32_t* idx = m.take<int32_t>(static_cast<size_t>(r2), &d_idx);
    if (m.overflow) return fail(c, RL_ERR_CAPACITY, "per-call metadata exceeds its workspace region");
    // rows [0, R1): prompts, K/V written to every slot of the group; rows
    // [R1, R): response tokens of each sequence, K/V written to its own slot
    // at positions P, P+1, ...  LM-head rows: each prompt's last row (it
    // scores response token 0 of every member), then response rows j < m-1
    // (row j scores token j+1).
    std::vector<Block> blocks;
    const int G = cf.n_q_heads / cf.n_kv_heads;
    const int tq = std::max(1, 16 / G);
    double kvpos = 0, scorepos = 0;
    int ns = 0, ni = 0;
    for (int p = 0; p < n_prompts; ++p) {
        const int b = prompt_offsets[p], len = prompt_offsets[p + 1] - b;
        const int shared_rows = shared_prompt_pages(c, len) * c->lay.page;
        for (int t = 0; t < len; ++t) {
            row_pos[b + t] = t;
            row_dst[b + t] = t < shared_rows ? -(slots[p * group] + 1) : p * group;
            row_slot[b + t] = slots[p * group];
        }
        for (int k = 0; k < group; ++k) dst[p * group + k] = slots[p * group + k];
        for (int t = 0; t < len; t += tq) blocks.push_back(Block{b + t, std::min(tq, len - t), slots[p * group], t});
        kvpos += len;
        scorepos += 0.5 * len * (len + 1.0);
        sel[ns] = b + len - 1;
        items[ns++] = ni;
        for (int k = 0; k < group; ++k) idx[ni++] = resp_offsets[p * group + k];
    }
    for (int p = 0; p < n_prompts; ++p) {
        const int P = prompt_offsets[p + 1] - prompt_offsets[p];
        for (int k = 0; k < group; ++k) {
            const int sq = p * group + k;
            const int o = resp_offsets[sq], mlen = resp_offsets[sq + 1] - o;
            const int b = R1 + o;
            for (int j = 0; j < mlen; ++j) {
                row_pos[b + j] = P + j;
                row_dst[b + j] = -(slots[sq] + 1);
                row_slot[b + j] = slots[sq];
            }
            for (int j = 0; j < mlen; j += tq) blocks.push_back(Block{b + j, std::min(tq, mlen - j), slots[sq], P + j});
            kvpos += P + mlen;
            scorepos += mlen * (P + 0.5 * (mlen + 1.0));
            for (int j = 0; j + 1 < mlen; ++j) {
                sel[ns] = b + j;
                items[ns++] = ni;
                idx[ni++] = o + j + 1;
            }
        }
    }
    items[ns] = ni;
    Fwd f;
    f.rows = R;
    f.tok = c->wsp<int32_t>(c->lay.off_tok);
    f.embeds = embeds;
    f.n_embed_rows = n_embed_rows;
    f.row_pos = d_row_pos;
    f.row_dst = d_row_dst;
    f.n_dst = group;
    f.dst_slots = d_dst;
    f.row_slot = d_row_slot;
    f.attn_kv_positions = kvpos;
    if (c->bf16() && c->opt_prefill_items) {
        const int C = choose_chunk(blocks, cf.n_kv_heads, c->opt_chunk, kPrefillChunk, c->lay.items_cap, false);
        st = build_items(c, &m, blocks, C, &f);
        if (st != RL_OK) return st;
    } else if (c->bf16()) {
        st = build_tiles(c, &m, blocks, &f);
        if (st != RL_OK) return st;
    } else {
        f.attn_score_positions = scorepos;
    }
    f.final_sel = d_sel;
    f.n_final = n_sel;
    // LM-head chunks: the fp32 logits go to the SwiGLU activation region when
    // it holds more rows than the logits buffer (it is free once the last
    // layer's down projection has run)
    const size_t mlp_rows = static_cast<size_t>(c->lay.R) * cf.ffn * c->lay.es / (4 * static_cast<size_t>(cf.vocab));
    if (mlp_rows > static_cast<size_t>(cf.max_seqs)) {
        f.logits = c->wsp<float>(c->lay.off_mlp);
        f.score_chunk = static_cast<int>(std::min<size_t>(mlp_rows, 1 << 20));
    } else {
        f.logits = c->wsp<float>(c->lay.off_logits);
        f.score_chunk = cf.max_seqs;
    }
    f.T = temperature > 0.0f ? temperature : 1.0f;
    f.out_logp = out_logp;
    f.score_items = d_items;
    f.score_idx = d_idx;
    f.score_targets = resp_tokens;
    set_group_pages(c, n_prompts, group, slots, plens, new_len);
    f.kvp = fill_pages(c, ps);
    st = upload_meta(c, &m, stage);
    if (st != RL_OK) return st;
    int32_t* tok = c->wsp<int32_t>(c->lay.off_tok);
    hipError_t e = hipMemcpyAsync(tok, prompt_tokens, sizeof(int32_t) * R1, hipMemcpyDeviceToDevice, c->stream);
    if (e == hipSuccess)
        e = hipMemcpyAsync(tok + R1, resp_tokens, sizeof(int32_t) * static_cast<size_t>(r2), hipMemcpyDeviceToDevice,
                           c->stream);
    if (e != hipSuccess) return hip_fail(c, e, "token copy");
    unshare(c, n_seq, slots);
    st = run_forward(c, f);
    std::vector<std::pair<int, int>> none;
    for (int i = 0; i < n_seq; ++i) {   // the slots were scratch
        c->len[slots[i]] = 0;
        none.emplace_back(slots[i], 0);
    }
    set_pages(c, none);   // a later call's K/V writes are ordered after this call's kernels
    return st;
}

rl_status rl_decode_step(rl_decode_ctx* ctx, int32_t n, const int32_t* slots, const uint64_t* seq_uids,
                         const int32_t* in_tok, const int32_t* forced_tok, const rl_sample_params* sp,
                         int32_t* out_tok, float* out_logp, float* out_logits) {
    if (!ctx_ok(ctx)) return RL_ERR_STATE;
    rl_decode_ctx* c = ctx;
    const rl_model_config& cf = c->cfg;
    if (n < 0) return fail(c, RL_ERR_INVALID_ARG, "n must be >= 0");
    if (n > cf.max_seqs) return fail(c, RL_ERR_CAPACITY, "n exceeds max_seqs");
    rl_status st = check_sp(c, sp);
    if (st != RL_OK) return st;
    if (n == 0) return RL_OK;
    if (!slots || !seq_uids || !in_tok || !out_tok || !out_logp)
        return fail(c, RL_ERR_INVALID_ARG, "required pointer is NULL");
    if (out_logits && !aligned(out_logits, 16)) return fail(c, RL_ERR_INVALID_ARG, "out_logits must be 16-byte aligned");
    std::vector<char> seen;
    st = check_slots(c, n, slots, &seen);
    if (st != RL_OK) return st;
    for (int i = 0; i < n; ++i)
        if (c->len[slots[i]] >= cf.max_ctx) return fail(c, RL_ERR_CAPACITY, "slot is full (length == max_ctx)");
    std::vector<std::pair<int, int>> want;
    if (c->paged()) {
        for (int i = 0; i < n; ++i) want.emplace_back(slots[i], c->len[slots[i]] + 1);
        if (!pages_fit(c, want)) return fail(c, RL_ERR_CAPACITY, "not enough free K/V pages");
    }
    DeviceGuard g(c->device);

    Meta m{};
    int stage = 0;
    st = begin_meta(c, &m, &stage);
    if (st != RL_OK) return st;
    const PageStage ps = take_pages(c, &m);
    int32_t *d_pos, *d_dst, *d_slot, *d_posn;
    uint64_t* d_uid;
    int32_t* pos = m.take<int32_t>(n, &d_pos);
    int32_t* dstr = m.take<int32_t>(n, &d_dst);
    int32_t* slot = m.take<int32_t>(n, &d_slot);
    int32_t* posn = m.take<int32_t>(n, &d_posn);
    uint64_t* uid = m.take<uint64_t>(n, &d_uid);
    if (m.overflow) return fail(c, RL_ERR_CAPACITY, "per-call metadata exceeds its workspace region");
    std::vector<Block> blocks(static_cast<size_t>(n));
    double kvpos = 0;
    for (int i = 0; i < n; ++i) {
        const int p = c->len[slots[i]];
        pos[i] = p;
        dstr[i] = i;
        slot[i] = slots[i];
        posn[i] = p + 1;
        uid[i] = seq_uids[i];
        blocks[i] = Block{i, 1, slots[i], p};
        const int src = c->opt_shared ? c->share_src[slots[i]] : -1;
        if (src >= 0) {   // a shared prompt: whole 32-position steps of it come from the group's first slot
            blocks[i].src = src;
            blocks[i].plen = c->share_len[slots[i]] / 32 * 32;
        }
        kvpos += p + 1;
    }
    Fwd f;
    f.rows = n;
    f.tok = in_tok;
    f.row_pos = d_pos;
    f.row_dst = d_dst;
    f.n_dst = 1;
    f.dst_slots = d_slot;
    f.row_slot = d_slot;
    f.attn_kv_positions = kvpos;
    f.attn_score_positions = kvpos;
    if (c->bf16()) {
        const int C = choose_chunk(blocks, cf.n_kv_heads, c->opt_chunk, 0, c->lay.items_cap, true);
        st = build_items(c, &m, blocks, C, &f);
        if (st != RL_OK) return st;
    }
    f.logits = out_logits ? out_logits : c->wsp<float>(c->lay.off_logits);
    f.n_out = n;
    f.uid = d_uid;
    f.pos_new = d_posn;
    f.forced = forced_tok;
    f.seed = sp->seed;
    f.T = sp->temperature;
    f.out_tok = out_tok;
    f.out_logp = out_logp;
    set_pages(c, want);
    f.kvp = fill_pages(c, ps);
    st = upload_meta(c, &m, stage);
    if (st != RL_OK) return st;
    st = run_forward(c, f);
    if (st != RL_OK) return st;
    for (int i = 0; i < n; ++i) c->len[slots[i]] += 1;
    c->plan.steps += 1;
    c->plan.items += f.plan_items;
    c->plan.shared_items += f.plan_shared;
    c->plan.pair_items += f.plan_pairs;
    c->plan.lds_workgroups += f.plan_lds;
    return RL_OK;
}

rl_status rl_sample_logits(rl_decode_ctx* ctx, int32_t n, const float* logits, const uint64_t* seq_uids,
                           const int32_t* pos_new, const int32_t* forced, const rl_sample_params* sp,
                           int32_t* out_tok, float* out_logp) {
    if (!ctx_ok(ctx)) return RL_ERR_STATE;
    rl_decode_ctx* c = ctx;
    if (n < 0) return fail(c, RL_ERR_INVALID_ARG, "n must be >= 0");
    if (n > c->cfg.max_seqs) return fail(c, RL_ERR_CAPACITY, "n exceeds max_seqs");
    rl_status st = check_sp(c, sp);
    if (st != RL_OK) return st;
    if (n == 0) return RL_OK;
    if (!logits || !seq_uids || !pos_new || !out_tok || !out_logp)
        return fail(c, RL_ERR_INVALID_ARG, "required pointer is NULL");
    if (!aligned(logits, 16)) return fail(c, RL_ERR_INVALID_ARG, "logits must be 16-byte aligned");
    for (int i = 0; i < n; ++i)
        if (pos_new[i] < 0) return fail(c, RL_ERR_INVALID_ARG, "pos_new must be >= 0");
    DeviceGuard g(c->device);
    Meta m{};
    int stage = 0;
    st = begin_meta(c, &m, &stage);
    if (st != RL_OK) return st;
    int32_t* d_posn;
    uint64_t* d_uid;
    int32_t* posn = m.take<int32_t>(n, &d_posn);
    uint64_t* uid = m.take<uint64_t>(n, &d_uid);
    if (m.overflow) return fail(c, RL_ERR_CAPACITY, "per-call metadata exceeds its workspace region");
    for (int i = 0; i < n; ++i) { posn[i] = pos_new[i]; uid[i] = seq_uids[i]; }
    st = upload_meta(c, &m, stage);
    if (st != RL_OK) return st;
    Prof pr(c, RL_K_SAMPLE);
    hipError_t e = launch_sample(logits, c->cfg.vocab, n, c->cfg.vocab, nullptr, d_uid, d_posn, forced, sp->seed,
                                 sp->temperature, c->sample_parts(), out_tok, out_logp,
                                 c->stream);
    if (e != hipSuccess) return hip_fail(c, e, "sample launch");
    pr.done(n * (c->cfg.vocab * 4.0 + 8.0), 0.0);
    return RL_OK;
}

rl_status rl_sample_logits_noalloc(int32_t n, int32_t vocab, const float* logits, int32_t ld,
                                   const uint64_t* seq_uids, const int32_t* pos_new, const int32_t* forced,
                                   const rl_sample_params* sp, int32_t* out_tok, float* out_logp, void* stream) {
    if (n < 0 || n > kNoAllocMaxRows) return RL_ERR_INVALID_ARG;
    if (vocab < 1 || vocab > (1 << 24) || vocab % 4 != 0 || ld < vocab || ld % 4 != 0) return RL_ERR_INVALID_ARG;
    if (!sp || sp->reserved != 0 || !(sp->temperature >= 0.0f) || !std::isfinite(sp->temperature))
        return RL_ERR_INVALID_ARG;
    if (n == 0) return RL_OK;
    if (!logits || !seq_uids || !pos_new || !out_tok || !out_logp) return RL_ERR_INVALID_ARG;
    if (!aligned(logits, 16)) return RL_ERR_INVALID_ARG;
    if (sample_parts_needed(n, vocab) > static_cast<size_t>(kStaticSampleParts)) return RL_ERR_CAPACITY;
    SamplePart* parts = nullptr;
    if (static_sample_parts(&parts) != hipSuccess) return RL_ERR_HIP;
    const hipError_t e = launch_sample(logits, ld, n, vocab, nullptr, seq_uids, pos_new, forced, sp->seed,
                                       sp->temperature, parts, out_tok, out_logp, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? RL_OK : RL_ERR_HIP;
}

namespace {

size_t kv_slot_packed_bytes(const rl_decode_ctx* c, int len) {
    const rl_model_config& cf = c->cfg;
    const size_t len8 = (static_cast<size_t>(len) + 7) / 8 * 8;
    return static_cast<size_t>(cf.n_layers) * cf.n_kv_heads * (len + len8) * cf.head_dim * c->lay.es;
}

// Offload (dir 0) or onload (dir 1) the packed live K/V of slots through the
// workspace staging region, a chunk of whole slots at a time.
rl_status kv_transfer(rl_decode_ctx* c, int dir, int n, const int32_t* slots, const int32_t* lens, uint8_t* host) {
    const rl_model_config& cf = c->cfg;
    const Layout& L = c->lay;
    size_t host_off = 0;
    int i0 = 0;
    while (i0 < n) {
        size_t bytes = 0;
        int i1 = i0;
        while (i1 < n && bytes + kv_slot_packed_bytes(c, lens[i1]) <= L.stage_bytes) bytes += kv_slot_packed_bytes(c, lens[i1++]);
        if (i1 == i0) return fail(c, RL_ERR_CAPACITY, "one slot's K/V exceeds the workspace staging region");
        Meta m{};
        int stage = 0;
        rl_status st = begin_meta(c, &m, &stage);
        if (st != RL_OK) return st;
        const PageStage ps = take_pages(c, &m);
        int32_t *d_slots, *d_lens;
        int64_t* d_base;
        int32_t* hs = m.take<int32_t>(i1 - i0, &d_slots);
        int32_t* hl = m.take<int32_t>(i1 - i0, &d_lens);
        int64_t* hb = m.take<int64_t>(i1 - i0, &d_base);
        if (m.overflow) return fail(c, RL_ERR_CAPACITY, "per-call metadata exceeds its workspace region");
        size_t b = 0;
        for (int i = i0; i < i1; ++i) {
            hs[i - i0] = slots[i];
            hl[i - i0] = lens[i];
            hb[i - i0] = static_cast<int64_t>(b);
            b += kv_slot_packed_bytes(c, lens[i]);
        }
        const KvPages kp = fill_pages(c, ps);
        st = upload_meta(c, &m, stage);
        if (st != RL_OK) return st;
        uint8_t* stg = c->ws + L.off_stage;
        hipError_t e = hipSuccess;
        if (dir == 1) e = hipMemcpyAsync(stg, host + host_off, bytes, hipMemcpyHostToDevice, c->stream);
        if (e == hipSuccess)
            e = launch_kv_pack(dir, d_slots, d_lens, d_base, i1 - i0, cf.n_layers, kp, cf.n_kv_heads,
                               cf.head_dim * L.es, L.es, c->kslab(), c->vslab(), stg, c->stream);
        if (e == hipSuccess && dir == 0) e = hipMemcpyAsync(host + host_off, stg, bytes, hipMemcpyDeviceToHost, c->stream);
        if (e != hipSuccess) return hip_fail(c, e, dir == 0 ? "KV offload" : "KV onload");
        host_off += bytes;
        i0 = i1;
    }
    return RL_OK;
}

}  // namespace

size_t rl_kv_offload_bytes(const rl_decode_ctx* ctx, int32_t n, const int32_t* slots) {
    if (!ctx_ok(ctx) || n < 0 || (n > 0 && !slots)) return 0;
    size_t total = 0;
    for (int i = 0; i < n; ++i) {
        if (slots[i] < 0 || slots[i] >= ctx->cfg.max_seqs) return 0;
        total += kv_slot_packed_bytes(ctx, ctx->len[slots[i]]);
    }
    return total;
}

rl_status rl_kv_offload(rl_decode_ctx* ctx, int32_t n, const int32_t* slots, void* host_dst, size_t host_bytes) {
    if (!ctx_ok(ctx)) return RL_ERR_STATE;
    rl_decode_ctx* c = ctx;
    if (n < 0) return fail(c, RL_ERR_INVALID_ARG, "n must be >= 0");
    if (n == 0) return RL_OK;
    if (!slots || !host_dst) return fail(c, RL_ERR_INVALID_ARG, "required pointer is NULL");
    std::vector<char> seen;
    rl_status st = check_slots(c, n, slots, &seen);
    if (st != RL_OK) return st;
    std::vector<int32_t> lens(static_cast<size_t>(n));
    size_t total = 0;
    for (int i = 0; i < n; ++i) {
        lens[i] = c->len[slots[i]];
        const size_t b = kv_slot_packed_bytes(c, lens[i]);
        if (b > c->lay.stage_bytes) return fail(c, RL_ERR_CAPACITY, "one slot's K/V exceeds the workspace staging region");
        total += b;
    }
    if (total > host_bytes) return fail(c, RL_ERR_CAPACITY, "host buffer smaller than rl_kv_offload_bytes");
    DeviceGuard g(c->device);
    return kv_transfer(c, 0, n, slots, lens.data(), static_cast<uint8_t*>(host_dst));
}

rl_status rl_kv_onload(rl_decode_ctx* ctx, int32_t n, const int32_t* slots, const int32_t* lengths,
                       const void* host_src, size_t host_bytes) {
    if (!ctx_ok(ctx)) return RL_ERR_STATE;
    rl_decode_ctx* c = ctx;
    if (n < 0) return fail(c, RL_ERR_INVALID_ARG, "n must be >= 0");
    if (n == 0) return RL_OK;
    if (!slots || !lengths || !host_src) return fail(c, RL_ERR_INVALID_ARG, "required pointer is NULL");
    std::vector<char> seen;
    rl_status st = check_slots(c, n, slots, &seen);
    if (st != RL_OK) return st;
    size_t total = 0;
    for (int i = 0; i < n; ++i) {
        if (lengths[i] < 0 || lengths[i] > c->cfg.max_ctx) return fail(c, RL_ERR_INVALID_ARG, "length out of range");
        const size_t b = kv_slot_packed_bytes(c, lengths[i]);
        if (b > c->lay.stage_bytes) return fail(c, RL_ERR_CAPACITY, "one slot's K/V exceeds the workspace staging region");
        total += b;
    }
    if (total > host_bytes) return fail(c, RL_ERR_CAPACITY, "host buffer smaller than the packed K/V of these lengths");
    // the slots' K/V is rewritten from position 0: new pages of their own
    const auto want = final_lengths(n, slots, lengths);
    if (!pages_fit(c, want, true)) return fail(c, RL_ERR_CAPACITY, "not enough free K/V pages");
    DeviceGuard g(c->device);
    set_pages(c, want, true);
    st = kv_transfer(c, 1, n, slots, lengths, static_cast<uint8_t*>(const_cast<void*>(host_src)));
    if (st != RL_OK) return st;
    for (int i = 0; i < n; ++i) c->len[slots[i]] = lengths[i];
    unshare(c, n, slots);
    return RL_OK;
}

rl_status rl_decode_rebind(rl_decode_ctx* ctx, const rl_weights* w, void* kv_pool, size_t kv_bytes,
                           void* workspace, size_t ws_bytes) {
    if (!ctx_ok(ctx)) return RL_ERR_STATE;
    rl_decode_ctx* c = ctx;
    if (!weights_ok(c->cfg, w)) return fail(c, RL_ERR_INVALID_ARG, "weights: NULL or misaligned pointer");
    if (!kv_pool || !workspace || !aligned(kv_pool, 256) || !aligned(workspace, 256))
        return fail(c, RL_ERR_INVALID_ARG, "KV pool and workspace must be 256-byte aligned device pointers");
    if (kv_bytes < c->lay.kv_bytes || ws_bytes < c->lay.ws_bytes) return fail(c, RL_ERR_CAPACITY, "buffer too small");
    DeviceGuard g(c->device);
    hipError_t e = hipStreamSynchronize(c->stream);   // nothing may still use the old buffers
    if (e != hipSuccess) return hip_fail(c, e, "rebind wait");
    c->w = *w;
    c->kv = static_cast<uint8_t*>(kv_pool);
    c->ws = static_cast<uint8_t*>(workspace);
    e = init_workspace(c);
    if (e != hipSuccess) return hip_fail(c, e, "rebind workspace setup");
    return RL_OK;
}

rl_status rl_release_slots(rl_decode_ctx* ctx, int32_t n, const int32_t* slots) {
    if (!ctx_ok(ctx)) return RL_ERR_STATE;
    if (n < 0 || (n > 0 && !slots)) return fail(ctx, RL_ERR_INVALID_ARG, "bad slot list");
    for (int i = 0; i < n; ++i)
        if (slots[i] < 0 || slots[i] >= ctx->cfg.max_seqs) return fail(ctx, RL_ERR_INVALID_ARG, "slot out of range");
    std::vector<std::pair<int, int>> none;
    for (int i = 0; i < n; ++i) {
        ctx->len[slots[i]] = 0;
        none.emplace_back(slots[i], 0);
    }
    set_pages(ctx, none);
    unshare(ctx, n, slots);
    return RL_OK;
}

rl_status rl_set_slot_lengths(rl_decode_ctx* ctx, int32_t n, const int32_t* slots, const int32_t* lengths) {
    if (!ctx_ok(ctx)) return RL_ERR_STATE;
    if (n < 0 || (n > 0 && (!slots || !lengths))) return fail(ctx, RL_ERR_INVALID_ARG, "bad slot list");
    for (int i = 0; i < n; ++i) {
        if (slots[i] < 0 || slots[i] >= ctx->cfg.max_seqs) return fail(ctx, RL_ERR_INVALID_ARG, "slot out of range");
        if (lengths[i] < 0 || lengths[i] > ctx->cfg.max_ctx) return fail(ctx, RL_ERR_INVALID_ARG, "length out of range");
    }
    const auto want = final_lengths(n, slots, lengths);
    // A length that ends inside a page the slot shares with others (its
    // group's prompt) takes a copy of that page: the slot's next K/V row goes
    // there.  (Counted before the call's pages are given back: conservative.)
    int64_t copies = 0;
    for (const auto& e : want) copies += shared_tail_page(ctx, e.first, e.second) >= 0;
    if (!pages_fit(ctx, want, false, copies)) return fail(ctx, RL_ERR_CAPACITY, "not enough free K/V pages");
    set_pages(ctx, want);
    const size_t mp = static_cast<size_t>(ctx->lay.maxp);
    for (const auto& e : want) {
        const int j = shared_tail_page(ctx, e.first, e.second);
        if (j < 0) continue;
        int32_t& pg = ctx->ptab[e.first * mp + j];
        const int32_t own = take_page(ctx, 1);
        DeviceGuard g(ctx->device);
        const hipError_t err = copy_page(ctx, pg, own);
        --ctx->pref[pg];
        pg = own;
        if (err != hipSuccess) return hip_fail(ctx, err, "K/V page copy");
    }
    for (int i = 0; i < n; ++i) ctx->len[slots[i]] = lengths[i];
    unshare(ctx, n, slots);
    return RL_OK;
}

int64_t rl_kv_free_pages(const rl_decode_ctx* ctx) {
    if (!ctx_ok(ctx) || !ctx->paged()) return -1;
    return static_cast<int64_t>(ctx->free_pages.size());
}

int32_t rl_slot_length(const rl_decode_ctx* ctx, int32_t slot) {
    if (!ctx_ok(ctx) || slot < 0 || slot >= ctx->cfg.max_seqs) return -1;
    return ctx->len[slot];
}

rl_status rl_decode_set_option(rl_decode_ctx* ctx, int32_t option, int64_t value) {
    if (!ctx_ok(ctx)) return RL_ERR_STATE;
    switch (option) {
        case RL_OPT_ATTN_CHUNK:
            if (value != 0 && (value < 32 || value > 65536 || value % 32 != 0))
                return fail(ctx, RL_ERR_INVALID_ARG, "attention chunk must be 0 or a multiple of 32 in [32, 65536]");
            ctx->opt_chunk = value;
            return RL_OK;
        case RL_OPT_GEMM_PLAN: {
            const int64_t k1 = value & 0xff, sp = (value >> 8) & 0xff, k2 = (value >> 16) & 0xff;
            const bool ok = value == 0 ||
                            (value >= 0 && (value >> 24) == 0 && k1 >= RL_GEMM_DIRECT && k1 <= RL_GEMM_GEMV_WIDE &&
                             sp <= kMaxSplits &&
                             (k2 == 0 || (k2 >= RL_GEMM_T128X256 && k2 <= RL_GEMM_T128_DEEP)));
            if (!ok) return fail(ctx, RL_ERR_INVALID_ARG, "invalid GEMM plan override");
            ctx->opt_gemm = value;
            return RL_OK;
        }
        case RL_OPT_PREFILL_ATTENTION:
            if (value != 0 && value != 1) return fail(ctx, RL_ERR_INVALID_ARG, "prefill attention option must be 0 or 1");
            ctx->opt_prefill_items = value == 1;
            return RL_OK;
        case RL_OPT_SHARED_PREFIX:
            if (value != 0 && value != 1) return fail(ctx, RL_ERR_INVALID_ARG, "shared prefix option must be 0 or 1");
            ctx->opt_shared = value == 1;
            return RL_OK;
        case RL_OPT_PROFILE:
            if (value < -1 || value >= (int64_t(1) << RL_K_COUNT))
                return fail(ctx, RL_ERR_INVALID_ARG, "profile must be a class bit mask or -1");
            ctx->profile = value == -1 ? ((1u << RL_K_COUNT) - 1u) : static_cast<uint32_t>(value);
            return RL_OK;
        default:
            return fail(ctx, RL_ERR_INVALID_ARG, "unknown option");
    }
}

rl_status rl_decode_tune_gemms(rl_decode_ctx* ctx, int32_t n_sizes, const int32_t* sizes) {
    if (!ctx_ok(ctx)) return RL_ERR_INVALID_ARG;
    if (n_sizes < 0 || n_sizes > 4096 || (n_sizes > 0 && !sizes))
        return fail(ctx, RL_ERR_INVALID_ARG, "n_sizes must be in [0, 4096] with a size array");
    if (ctx->cfg.n_experts > 0 && n_sizes > 0)
        return fail(ctx, RL_ERR_UNSUPPORTED, "measured GEMM plans cover dense models (the experts have their own kernel)");
    std::vector<int> v(sizes, sizes + n_sizes);
    for (int i = 0; i < n_sizes; ++i) {
        if (v[i] < 1 || v[i] > ctx->cfg.max_seqs)
            return fail(ctx, RL_ERR_INVALID_ARG, "batch sizes must be in [1, max_seqs]");
        if (i > 0 && v[i] <= v[i - 1]) return fail(ctx, RL_ERR_INVALID_ARG, "batch sizes must be increasing");
    }
    if (n_sizes > 0 && !ctx->bf16()) return fail(ctx, RL_ERR_UNSUPPORTED, "GEMM plans are tuned for bf16 models only");
    for (int32_t l : ctx->len)
        if (l != 0) return fail(ctx, RL_ERR_INVALID_ARG, "GEMM plans are measured with no live sequence (every length 0)");
    ctx->tuned.clear();
    if (n_sizes == 0) return RL_OK;
    DeviceGuard g(ctx->device);
    return tune_gemms(ctx, v);
}

rl_status rl_decode_gemm_plan(rl_decode_ctx* ctx, int32_t kclass, int32_t rows, int64_t* plan_code,
                              float* tuned_us) {
    if (!ctx_ok(ctx)) return RL_ERR_INVALID_ARG;
    if (kclass != RL_K_GEMM_QKV && kclass != RL_K_GEMM_O && kclass != RL_K_GEMM_GATE_UP &&
        kclass != RL_K_GEMM_DOWN && kclass != RL_K_GEMM_LM_HEAD)
        return fail(ctx, RL_ERR_INVALID_ARG, "kclass must be a GEMM class");
    if (rows < 1 || rows > std::max(ctx->cfg.max_seqs, ctx->cfg.max_prefill_tokens))
        return fail(ctx, RL_ERR_INVALID_ARG, "rows out of range");
    if (!plan_code) return fail(ctx, RL_ERR_INVALID_ARG, "plan_code is NULL");
    if (!ctx->bf16()) return fail(ctx, RL_ERR_UNSUPPORTED, "GEMM plans exist for bf16 models only");
    const rl_model_config& cf = ctx->cfg;
    const int H = cf.hidden, F = cf.ffn, HqD = cf.n_q_heads * cf.head_dim;
    int Nw = cf.vocab, K = H, epi = EPI_F32;
    if (kclass == RL_K_GEMM_QKV) Nw = ctx->lay.nqkv;
    if (kclass == RL_K_GEMM_O) { Nw = H; K = HqD; epi = EPI_RESID; }
    if (kclass == RL_K_GEMM_GATE_UP) { Nw = 2 * F; epi = EPI_SWIGLU; }
    if (kclass == RL_K_GEMM_DOWN) { Nw = H; K = F; epi = EPI_RESID; }
    GemmPlan p;
    float us = -1.0f;
    if (!(ctx->opt_gemm != 0 && plan_gemm_forced(rows, Nw, K, epi, F, ctx->opt_gemm, &p)) &&
        !tuned_plan(ctx, kclass, rows, Nw, K, epi, &p, &us))
        p = plan_gemm_bf16(rows, Nw, K, epi, F);
    *plan_code = gemm_plan_code_of(p);
    if (tuned_us) *tuned_us = us;
    return RL_OK;
}

rl_status rl_decode_kernel_stats(rl_decode_ctx* ctx, int32_t kclass, rl_kernel_stats* out) {
    if (!ctx_ok(ctx)) return RL_ERR_STATE;
    if (kclass < 0 || kclass >= RL_K_COUNT || !out) return fail(ctx, RL_ERR_INVALID_ARG, "bad kernel class");
    DeviceGuard g(ctx->device);
    hipError_t e = harvest(ctx);
    if (e != hipSuccess) return hip_fail(ctx, e, "profile harvest");
    *out = ctx->stats[kclass];
    return RL_OK;
}

rl_status rl_decode_attn_plan_stats(const rl_decode_ctx* ctx, rl_attn_plan_stats* out) {
    if (!ctx_ok(ctx)) return RL_ERR_STATE;
    if (!out) return RL_ERR_INVALID_ARG;
    *out = ctx->plan;
    return RL_OK;
}

rl_status rl_decode_reset_stats(rl_decode_ctx* ctx) {
    if (!ctx_ok(ctx)) return RL_ERR_STATE;
    DeviceGuard g(ctx->device);
    hipError_t e = harvest(ctx);
    if (e != hipSuccess) return hip_fail(ctx, e, "profile harvest");
    for (int i = 0; i < RL_K_COUNT; ++i) {
        ctx->stats[i].launches = 0;
        ctx->stats[i].total_ms = 0;
        ctx->stats[i].alg_bytes = 0;
        ctx->stats[i].alg_flops = 0;
    }
    ctx->plan = rl_attn_plan_stats{};
    return RL_OK;
}

rl_status rl_probe_gumbel_bound(uint32_t lo, uint64_t count, int32_t n_blocks, uint32_t* viol, float* min_margin,
                                void* stream) {
    if (!viol || !min_margin || n_blocks < 1 || n_blocks > 65536) return RL_ERR_INVALID_ARG;
    if (count == 0 || count > (1ull << 32) || lo + (count - 1) > 0xFFFFFFFFull) return RL_ERR_INVALID_ARG;
    if (!aligned(viol, 4) || !aligned(min_margin, 4)) return RL_ERR_INVALID_ARG;
    return launch_gumbel_bound_probe(lo, count, n_blocks, viol, min_margin, static_cast<hipStream_t>(stream)) ==
                   hipSuccess
               ? RL_OK
               : RL_ERR_HIP;
}

rl_status rl_probe_copy(void* dst, const void* src, size_t bytes, void* stream) {
    if (!dst || !src || bytes % 16 || !aligned(dst, 16) || !aligned(src, 16)) return RL_ERR_INVALID_ARG;
    hipError_t e = launch_copy16(dst, src, bytes / 16, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? RL_OK : RL_ERR_HIP;
}

rl_status rl_probe_read(const void* src, size_t bytes, int32_t n_blocks, uint32_t* out, void* stream) {
    if (!src || !out || bytes % 16 || !aligned(src, 16) || n_blocks < 1 || n_blocks > 65536)
        return RL_ERR_INVALID_ARG;
    hipError_t e = launch_read16(src, bytes / 16, out, n_blocks, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? RL_OK : RL_ERR_HIP;
}

rl_status rl_probe_mfma(int32_t n_blocks, int32_t iters, float* out, void* stream) {
    if (!out || n_blocks < 1 || n_blocks > 65536 || iters < 1 || iters > (1 << 20)) return RL_ERR_INVALID_ARG;
    hipError_t e = launch_mfma_probe(n_blocks, iters, out, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? RL_OK : RL_ERR_HIP;
}

}  // extern "C"
