// Host engine and C ABI of the refinement-step library (see include/dlm.h).
//
// The engine lays the synthetic weights out in the caller's device buffer,
// carves the caller's workspace, and enqueues the kernel sequence of one
// refinement pass on the caller's stream:
//   embed -> L x [rmsnorm, QKV GEMM (+RoPE), attention, O GEMM (+residual),
//                 rmsnorm, FFN (dense SwiGLU, or router/top-k/dispatch/grouped
//                 expert GEMMs/combine)]
//         -> final rmsnorm of draft rows -> LM-head GEMM with fused softmax
//            partials -> merge -> threshold edit.
// Block-AR drafting runs the same layer sequence over one window of rows at a
// time (the prompt, or one block), with K and V kept per layer in a cache that
// spans the whole sequence.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <chrono>
#include <mutex>
#include <atomic>
#include <exception>
#include <new>
#include <string>
#include <vector>

#include "../../include/dlm.h"
#include "kernels.h"

namespace {

thread_local std::string g_last_error;

dlm_status fail(dlm_status s, const std::string& msg) {
    g_last_error = msg;
    return s;
}

// No C++ exception leaves an entry point: each catches what its body throws
// (a failed host allocation in a plan's vectors, a message string or the
// profiling records) and reports it as a status.  The message is set without
// allocating when the string already holds enough capacity.
void set_error_noexcept(const char* msg) noexcept {
    try {
        g_last_error.assign(msg);
    } catch (...) {
        g_last_error.clear();
    }
}

dlm_status caught_exception() noexcept {
    try {
        throw;
    } catch (const std::bad_alloc&) {
        set_error_noexcept("a host memory allocation failed");
        return DLM_ERR_NO_MEMORY;
    } catch (const std::exception& e) {
        set_error_noexcept(e.what());
    } catch (...) {
        set_error_noexcept("unexpected exception");
    }
    return DLM_ERR_INTERNAL;
}

// Test hook: the n-th pass through a host allocation point from now throws
// std::bad_alloc (0: never).
std::atomic<int> g_fail_alloc_in{0};

void alloc_point() {
    int v = g_fail_alloc_in.load(std::memory_order_relaxed);
    while (v > 0 && !g_fail_alloc_in.compare_exchange_weak(v, v - 1, std::memory_order_relaxed)) {
    }
    if (v == 1) throw std::bad_alloc();
}

#define HIP_TRY(expr)                                                                         \
    do {                                                                                      \
        hipError_t _e = (expr);                                                               \
        if (_e != hipSuccess)                                                                 \
            return fail(DLM_ERR_HIP, std::string(#expr) + ": " + hipGetErrorString(_e));     \
    } while (0)

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Tensor kinds (layer_field 0: embedding 0, LM head 1).
enum { K_WQ = 0, K_WK, K_WV, K_WO, K_FG, K_FU, K_FD, K_ROUTER, K_EG, K_EU, K_ED, K_SG, K_SU, K_SD };

uint32_t tensor_id(int layer_field, int kind, int expert) {
    return ((uint32_t)layer_field << 20) | ((uint32_t)kind << 12) | (uint32_t)expert;
}

struct TensorInit {
    size_t off;          // byte offset in the weight buffer
    uint64_t n_phys;     // physical elements
    uint32_t cols;
    uint32_t tid_a, tid_b;
    int layout;          // 0 plain, 1 gate/up interleaved in 32-row blocks
    float scale;         // lm_head_scale for the LM head, else 1
    int kind_fill;       // 1: fill with 1.0 (norm gains) instead of random
};

struct LayerPtrs {
    size_t wqkv, wo, g1, g2, wgu, wd, wr;
};

struct WeightPlan {
    size_t total = 0;
    size_t emb = 0, lm = 0, gf = 0;
    std::vector<LayerPtrs> layers;
    std::vector<TensorInit> inits;
};

std::string validate(const dlm_config* c) {
    if (!c) return "config is NULL";
    if (c->n_layers < 0) return "n_layers < 0";
    if (c->d_model <= 0 || c->d_model % 128) return "d_model must be a positive multiple of 128";
    if (c->head_dim != 64 && c->head_dim != 128) return "head_dim must be 64 or 128";
    if (c->n_heads <= 0 || c->n_kv_heads <= 0 || c->n_heads % c->n_kv_heads)
        return "n_heads must be a positive multiple of n_kv_heads";
    if ((c->n_heads * c->head_dim) % 128 || (c->n_kv_heads * c->head_dim) % 128)
        return "n_heads*head_dim and n_kv_heads*head_dim must be multiples of 128";
    if (c->vocab < 2) return "vocab must be >= 2";
    if (c->mask_id < 0 || c->mask_id >= c->vocab) return "mask_id out of range";
    if (c->n_experts < 0 || c->n_experts > 256) return "n_experts must be in [0, 256]";
    if (c->n_experts == 0) {
        if (c->ffn_dim <= 0 || c->ffn_dim % 64) return "ffn_dim must be a positive multiple of 64";
    } else {
        if (c->top_k < 1 || c->top_k > 8 || c->top_k > c->n_experts) return "top_k must be in [1, min(8, n_experts)]";
        if (c->expert_ffn_dim <= 0 || c->expert_ffn_dim % 64) return "expert_ffn_dim must be a positive multiple of 64";
        if (c->n_shared_experts < 0 || c->n_shared_experts > 1) return "n_shared_experts must be 0 or 1";
    }
    if (!(c->norm_eps >= 0.f) || !isfinite(c->norm_eps)) return "norm_eps must be finite and >= 0";
    if (!(c->rope_theta > 0.f) || !isfinite(c->rope_theta)) return "rope_theta must be finite and > 0";
    if (!isfinite(c->init_std) || !isfinite(c->lm_head_scale)) return "init_std / lm_head_scale must be finite";
    return "";
}

WeightPlan plan_weights(const dlm_config& c) {
    alloc_point();
    WeightPlan p;
    const int d = c.d_model, hd = c.head_dim, H = c.n_heads, KV = c.n_kv_heads;
    auto add = [&](uint64_t elems) {
        const size_t off = p.total;
        p.total = align_up(p.total + elems * 2);
        return off;
    };
    auto plain = [&](size_t off, uint64_t rows, uint32_t cols, uint32_t tid, float scale) {
        p.inits.push_back(TensorInit{off, rows * cols, cols, tid, tid, 0, scale, 0});
    };
    auto inter = [&](size_t off, uint64_t f, uint32_t cols, uint32_t tg, uint32_t tu) {
        p.inits.push_back(TensorInit{off, 2 * f * cols, cols, tg, tu, 1, 1.f, 0});
    };
    auto ones = [&](size_t off, uint64_t n) {
        p.inits.push_back(TensorInit{off, n, (uint32_t)n, 0, 0, 0, 1.f, 1});
    };
    p.emb = add((uint64_t)c.vocab * d);
    plain(p.emb, c.vocab, d, tensor_id(0, 0, 0), 1.f);
    p.lm = add((uint64_t)c.vocab * d);
    plain(p.lm, c.vocab, d, tensor_id(0, 1, 0), c.lm_head_scale);
    p.gf = add(d);
    ones(p.gf, d);
    for (int l = 0; l < c.n_layers; ++l) {
        const int f = l + 1;
        LayerPtrs L{};
        const uint64_t nq = (uint64_t)H * hd, nk = (uint64_t)KV * hd;
        L.wqkv = add((nq + 2 * nk) * d);
        plain(L.wqkv, nq, d, tensor_id(f, K_WQ, 0), 1.f);
        plain(L.wqkv + nq * d * 2, nk, d, tensor_id(f, K_WK, 0), 1.f);
        plain(L.wqkv + (nq + nk) * d * 2, nk, d, tensor_id(f, K_WV, 0), 1.f);
        L.wo = add((uint64_t)d * nq);
        plain(L.wo, d, (uint32_t)nq, tensor_id(f, K_WO, 0), 1.f);
        L.g1 = add(d);
        ones(L.g1, d);
        L.g2 = add(d);
        ones(L.g2, d);
        if (c.n_experts == 0) {
            const uint64_t F = c.ffn_dim;
            L.wgu = add(2 * F * d);
            inter(L.wgu, F, d, tensor_id(f, K_FG, 0), tensor_id(f, K_FU, 0));
            L.wd = add((uint64_t)d * F);
            plain(L.wd, d, (uint32_t)F, tensor_id(f, K_FD, 0), 1.f);
            L.wr = 0;
        } else {
            const uint64_t F = c.expert_ffn_dim;
            const int G = c.n_experts + c.n_shared_experts;
            L.wr = add((uint64_t)c.n_experts * d);
            plain(L.wr, c.n_experts, d, tensor_id(f, K_ROUTER, 0), 1.f);
            L.wgu = add((uint64_t)G * 2 * F * d);
            for (int e = 0; e < G; ++e) {
                const bool sh = e >= c.n_experts;
                const int ei = sh ? e - c.n_experts : e;
                inter(L.wgu + (uint64_t)e * 2 * F * d * 2, F, d, tensor_id(f, sh ? K_SG : K_EG, ei),
                      tensor_id(f, sh ? K_SU : K_EU, ei));
            }
            L.wd = add((uint64_t)G * d * F);
            for (int e = 0; e < G; ++e) {
                const bool sh = e >= c.n_experts;
                const int ei = sh ? e - c.n_experts : e;
                plain(L.wd + (uint64_t)e * d * F * 2, d, (uint32_t)F, tensor_id(f, sh ? K_SD : K_ED, ei), 1.f);
            }
        }
        p.layers.push_back(L);
    }
    return p;
}

// Workspace carve-up for one (B, P, D).
struct Workspace {
    size_t total = 0;
    size_t x, h, q, k, v, attn, rope, hf, ids, wts, grp_off, tile_tab,
        n_tiles, slot, a_rows, ecount, hexp, y, hfin, partials, top1, conf, maxlogit, counters, tokens;
    int rows_total = 0, max_tiles = 0, n_vtiles = 0;
};

constexpr int kExpertBM = 256, kExpertBN = 256;
constexpr int kHeadBM = 256, kHeadBN = 256;

Workspace plan_workspace(const dlm_config& c, int B, int P, int D) {
    Workspace w;
    const int64_t S = P + D, T = (int64_t)B * S, R = (int64_t)B * D;
    const int d = c.d_model, hd = c.head_dim;
    auto add = [&](int64_t bytes) {
        const size_t off = w.total;
        w.total = align_up(w.total + (size_t)std::max<int64_t>(bytes, 1));
        return off;
    };
    w.x = add(T * d * 4);
    w.h = add(T * d * 2);
    w.q = add((int64_t)B * c.n_heads * S * hd * 2);
    w.k = add(((int64_t)B * c.n_kv_heads * S + 64) * hd * 2);         // + one 64-key tile of tail
    w.v = add((int64_t)B * c.n_kv_heads * hd * vt_stride((int)S) * 2);   // V^T, rows padded to tiles
    w.attn = add(T * c.n_heads * hd * 2);
    w.rope = add(S * (hd / 2) * 8);
    if (c.n_experts == 0) {
        w.hf = add(T * c.ffn_dim * 2);
    } else {
        const int E = c.n_experts, k = c.top_k, G = E + c.n_shared_experts;
        w.rows_total = (int)(T * k + T * c.n_shared_experts);
        w.max_tiles = (w.rows_total + kExpertBM - 1) / kExpertBM + G;
        w.ids = add(T * k * 4);
        w.wts = add(T * k * 4);
        w.grp_off = add((G + 1) * 4);
        w.tile_tab = add((int64_t)w.max_tiles * 8);
        w.n_tiles = add(4);
        w.slot = add(T * k * 4);
        w.a_rows = add((int64_t)w.rows_total * 4);
        w.ecount = add((T + 31) / 32 * E * 4);           // per router workgroup and expert counts
        w.hexp = add((int64_t)w.rows_total * c.expert_ffn_dim * 2);
        w.y = add((int64_t)w.rows_total * d * 2);
    }
    w.n_vtiles = 2 * ((c.vocab + kHeadBM - 1) / kHeadBM);   // LM-head partials per half tile
    w.hfin = add(R * d * 2);
    w.partials = add((int64_t)w.n_vtiles * R * 16);
    w.top1 = add(R * 4);
    w.conf = add(R * 4);
    w.maxlogit = add(R * 4);
    w.counters = add(CNT_WORDS * 4);                   // pass counters (PassCounter)
    w.tokens = add(T * 4);
    return w;
}

std::string check_shape(int B, int P, int D) {
    if (B <= 0) return "batch must be > 0";
    if (P < 0) return "prompt_len must be >= 0";
    if (D <= 0) return "draft_len must be > 0";
    const int64_t S = (int64_t)P + D;
    if (S > 65536 || (int64_t)B * S > (1 << 26)) return "batch * seq_len too large";
    return "";
}

// The kernels address the [tokens][d_model] and [tokens][heads * head_dim]
// activations through 32-bit buffer offsets: such a buffer must stay below 2 GiB.
std::string check_offsets(const dlm_config& c, int64_t T) {
    const int64_t width = std::max<int64_t>(c.d_model, (int64_t)c.n_heads * c.head_dim);
    if (T * width * 2 >= ((int64_t)1 << 31)) return "batch * seq_len * d_model too large (2 GiB activation buffers)";
    return "";
}

struct ProfRec {
    const char* name;
    hipEvent_t a, b;
};

}  // namespace

struct dlm_model {
    dlm_config cfg;
    uint64_t seed;
    int device = 0;              // device current at set-up (holds the weights)
    char* scratch = nullptr;     // that device's copy of the static scratch array
    char* base;
    size_t bytes;
    WeightPlan plan;
    // profiling
    std::string prof_filter;
    bool prof_on = false;
    std::vector<ProfRec> prof;
    size_t prof_used = 0;
};

namespace {

struct Ctx {
    dlm_model* m;
    const dlm_config& c;
    char* ws;
    Workspace w;
    hipStream_t st;
    int B, P, D, S, T, R;
    bool h_ready = false;           // h already holds the next block's normalised input
    int pos_shift = 0;              // draft positions are P + shift + i (a span refined on its own)
    // Drafting windows: the S rows of each sequence are positions q0 .. q0+S-1
    // of a sequence of kv_seq positions whose K / V^T live in the per-layer
    // caches kc / vc (kv_seq = 0: refinement, K and V^T of the S rows only).
    int q0 = 0, kv_seq = 0;
    bf16_t* kc = nullptr;
    bf16_t* vc = nullptr;
    size_t kc_layer = 0, vc_layer = 0;  // elements per layer
    const float2* rope_all = nullptr;   // RoPE table of all kv_seq positions
    bool kv_only = false;               // stop after the last layer's K/V (cache commit)
    bool no_events = false;             // no profiling events (the entry point allocates nothing)
    int att_split = 0, att_keys_lo = 0;  // window rows below att_split see only att_keys_lo keys
    float* dbg_router_logits = nullptr;  // test hook: router logits [T][E] of the layer run
    // Only the draft rows leave the last block (the head reads nothing else):
    // its MoE FFN then runs on the B*D draft rows alone.  Their K / V for the
    // block's attention come from the QKV projection of every row, as before.
    bool draft_rows_last_ffn = false;
    template <class Tp>
    Tp* at(size_t off) const { return reinterpret_cast<Tp*>(ws + off); }
    const bf16_t* wt(size_t off) const { return reinterpret_cast<const bf16_t*>(m->base + off); }
};

// Profiling: HIP events around launches of kernels whose name matches the filter.
void prof_begin(Ctx& x, const char* name) {
    dlm_model* m = x.m;
    if (!m->prof_on || x.no_events) return;
    if (!(m->prof_filter == "*" || m->prof_filter == name)) return;
    if (m->prof_used == m->prof.size()) {
        alloc_point();
        if (m->prof.size() == m->prof.capacity())   // may throw: before the events exist
            m->prof.reserve(2 * m->prof.size() + 64);
        ProfRec r{name, nullptr, nullptr};
        if (hipEventCreate(&r.a) != hipSuccess) return;
        if (hipEventCreate(&r.b) != hipSuccess) {
            (void)hipEventDestroy(r.a);
            return;
        }
        m->prof.push_back(r);
    }
    ProfRec& r = m->prof[m->prof_used];
    r.name = name;
    hipEventRecord(r.a, x.st);
}
void prof_end(Ctx& x, const char* name) {
    dlm_model* m = x.m;
    if (!m->prof_on || x.no_events) return;
    if (!(m->prof_filter == "*" || m->prof_filter == name)) return;
    if (m->prof_used >= m->prof.size()) return;
    hipEventRecord(m->prof[m->prof_used].b, x.st);
    ++m->prof_used;
}

#define LAUNCH(ctx, name, call)          \
    do {                                 \
        prof_begin(ctx, name);           \
        call;                            \
        prof_end(ctx, name);             \
    } while (0)

dlm_status gemm(Ctx& x, const char* name, const GemmArgs& a, int epi, bool grouped, int bm, int bn,
                int max_tiles) {
    hipError_t e;
    prof_begin(x, name);
    e = launch_gemm(a, epi, grouped, bm, bn, max_tiles, x.st);
    prof_end(x, name);
    if (e != hipSuccess) return fail(DLM_ERR_HIP, std::string("gemm ") + name + ": " + hipGetErrorString(e));
    return DLM_OK;
}

GemmArgs gemm_args(const bf16_t* A, int64_t lda, const bf16_t* B, int64_t ldb, int M, int N, int K) {
    GemmArgs a;
    memset(&a, 0, sizeof(a));
    a.A = A;
    a.lda = lda;
    a.B = B;
    a.ldb = ldb;
    a.M = M;
    a.N = N;
    a.K = K;
    a.group_m = 4;
    return a;
}

#define TRY(expr)                        \
    do {                                 \
        dlm_status _s = (expr);          \
        if (_s != DLM_OK) return _s;     \
    } while (0)

// One transformer block on the fp32 residual stream x (in place).
dlm_status run_layer(Ctx& x, int l) {
    const dlm_config& c = x.c;
    const LayerPtrs& L = x.m->plan.layers[l];
    const int d = c.d_model, hd = c.head_dim, H = c.n_heads, KV = c.n_kv_heads;
    float* xs = x.at<float>(x.w.x);
    bf16_t* h = x.at<bf16_t>(x.w.h);
    bf16_t* q = x.at<bf16_t>(x.w.q);
    bf16_t* k = x.kc ? x.kc + (size_t)l * x.kc_layer : x.at<bf16_t>(x.w.k);
    bf16_t* v = x.vc ? x.vc + (size_t)l * x.vc_layer : x.at<bf16_t>(x.w.v);
    bf16_t* attn = x.at<bf16_t>(x.w.attn);
    const int kvS = x.kv_seq ? x.kv_seq : x.S;

    if (!x.h_ready) LAUNCH(x, "rmsnorm", launch_rmsnorm(xs, x.wt(L.g1), h, x.T, d, c.norm_eps, x.st));
    x.h_ready = false;
    {
        // Transposed: rows = the (H + 2 KV) * hd output features, columns = tokens.
        const int N = (H + 2 * KV) * hd;
        GemmArgs a = gemm_args(x.wt(L.wqkv), d, h, d, N, x.T, d);
        a.q = q;
        a.k = k;
        a.v = v;
        a.rope = x.rope_all ? x.rope_all : x.at<float2>(x.w.rope);
        a.seq = x.S;
        a.kv_seq = kvS;
        a.pos0 = x.q0;
        a.n_heads = H;
        a.n_kv = KV;
        a.head_dim = hd;
        const int64_t big_tiles = (int64_t)((N + 255) / 256) * ((x.T + 255) / 256);
        a.variant = big_tiles >= 192 ? 11 : 0;          // ping-pong 8-wave 256x256 tiles
        TRY(gemm(x, "gemm_qkv", a, EPI_QKV, false, 256, a.variant != 0 ? 256 : 128, 0));
    }
    if (x.kv_only && l + 1 == c.n_layers) return DLM_OK;    // the cache holds this window's K/V now
    {
        prof_begin(x, "attention");
        hipError_t e = launch_attention(q, k, v, attn, x.B, x.S, kvS, x.q0 + x.S, H, KV, hd, x.st, x.att_split,
                                        x.att_keys_lo);
        prof_end(x, "attention");
        if (e != hipSuccess) return fail(DLM_ERR_HIP, std::string("attention: ") + hipGetErrorString(e));
    }
    {
        GemmArgs a = gemm_args(attn, (int64_t)H * hd, x.wt(L.wo), (int64_t)H * hd, x.T, d, H * hd);
        a.out = xs;
        a.ldo = d;
        const int64_t big_tiles = (int64_t)((x.T + 255) / 256) * ((d + 255) / 256);
        a.variant = big_tiles >= 128 ? 11 : 0;
        // up to 1024 rows (drafting windows): 128 x 64 tiles, twice the workgroups of 128 x 128
        const int obm = a.variant != 0 || x.T >= 4096 ? 256 : 128;
        const int obn = a.variant != 0 ? 256 : x.T <= 1024 ? 64 : 128;
        TRY(gemm(x, "gemm_o", a, EPI_RESID, false, obm, obn, 0));
    }
    // MoE FFN of the last block on the draft rows only (rows in [B][D] order)
    const bool draft_ffn = x.draft_rows_last_ffn && l + 1 == c.n_layers && c.n_experts > 0 && x.P > 0;
    const int Tf = draft_ffn ? x.R : x.T;
    if (draft_ffn)
        LAUNCH(x, "rmsnorm", launch_rmsnorm_draft_rows(xs, x.wt(L.g2), h, x.B, x.S, x.P, x.D, d, c.norm_eps, x.st));
    else
        LAUNCH(x, "rmsnorm", launch_rmsnorm(xs, x.wt(L.g2), h, x.T, d, c.norm_eps, x.st));
    if (c.n_experts == 0) {
        const int F = c.ffn_dim;
        bf16_t* hf = x.at<bf16_t>(x.w.hf);
        GemmArgs a = gemm_args(h, d, x.wt(L.wgu), d, x.T, 2 * F, d);
        a.out = hf;
        a.ldo = F;
        TRY(gemm(x, "gemm_ffn_gate_up", a, EPI_SWIGLU, false, x.T >= 4096 ? 256 : 128, 256, 0));
        GemmArgs b = gemm_args(hf, F, x.wt(L.wd), F, x.T, d, F);
        b.out = xs;
        b.ldo = d;
        TRY(gemm(x, "gemm_ffn_down", b, EPI_RESID, false, x.T >= 4096 ? 256 : 128, 128, 0));
        return DLM_OK;
    }
    const int E = c.n_experts, kk = c.top_k, NS = c.n_shared_experts, F = c.expert_ffn_dim;
    int32_t* ids = x.at<int32_t>(x.w.ids);
    float* wts = x.at<float>(x.w.wts);
    int32_t* grp_off = x.at<int32_t>(x.w.grp_off);
    int2* tile_tab = x.at<int2>(x.w.tile_tab);
    int32_t* n_tiles = x.at<int32_t>(x.w.n_tiles);
    int32_t* slot = x.at<int32_t>(x.w.slot);
    int32_t* a_rows = x.at<int32_t>(x.w.a_rows);
    int32_t* wg_counts = x.at<int32_t>(x.w.ecount);
    bf16_t* hexp = x.at<bf16_t>(x.w.hexp);
    bf16_t* y = x.at<bf16_t>(x.w.y);
    {
        prof_begin(x, "router_topk");
        hipError_t e = launch_router_topk(h, x.wt(L.wr), Tf, d, E, kk, ids, wts, slot, wg_counts, x.st,
                                          x.dbg_router_logits);
        prof_end(x, "router_topk");
        if (e != hipSuccess) return fail(DLM_ERR_HIP, std::string("router_topk: ") + hipGetErrorString(e));
        prof_begin(x, "dispatch");
        e = launch_dispatch(ids, Tf, kk, E, NS, kExpertBM, wg_counts, grp_off, tile_tab, n_tiles, slot, a_rows,
                            x.st);
        prof_end(x, "dispatch");
        if (e != hipSuccess) return fail(DLM_ERR_HIP, std::string("dispatch: ") + hipGetErrorString(e));
    }
    {
        GemmArgs a = gemm_args(h, d, x.wt(L.wgu), d, 0, 2 * F, d);
        a.b_group_stride = (int64_t)2 * F * d;
        a.tile_tab = tile_tab;
        a.n_tiles = n_tiles;
        a.grp_off = grp_off;
        a.a_rows = a_rows;
        a.out = hexp;
        a.ldo = F;
        a.variant = 11;                                 // ping-pong, third stage for the streamed expert weights (B)
        TRY(gemm(x, "gemm_expert_gate_up", a, EPI_SWIGLU, true, kExpertBM, kExpertBN, x.w.max_tiles));
    }
    {
        GemmArgs a = gemm_args(hexp, F, x.wt(L.wd), F, 0, d, F);
        a.b_group_stride = (int64_t)d * F;
        a.tile_tab = tile_tab;
        a.n_tiles = n_tiles;
        a.grp_off = grp_off;
        a.a_rows = nullptr;
        a.out = y;
        a.ldo = d;
        a.variant = 11;
        TRY(gemm(x, "gemm_expert_down", a, EPI_BF16, true, kExpertBM, kExpertBN, x.w.max_tiles));
    }
    // The combine also normalises each finished row for the next block.
    const bool fuse = l + 1 < c.n_layers;
    LAUNCH(x, "combine", launch_combine(xs, y, slot, wts, grp_off, Tf, kk, E, NS, d,
                                        fuse ? x.wt(x.m->plan.layers[l + 1].g1) : nullptr, h, c.norm_eps, x.st,
                                        draft_ffn ? x.S : 0, draft_ffn ? x.P : 0, draft_ffn ? x.D : 0));
    x.h_ready = fuse;
    return DLM_OK;
}

dlm_status run_prologue(Ctx& x, const int32_t* tokens) {
    const dlm_config& c = x.c;
    LAUNCH(x, "rope_table", launch_rope_table(x.at<float2>(x.w.rope), x.S, c.head_dim / 2, (double)c.rope_theta, x.P,
                                              x.pos_shift, x.st));
    LAUNCH(x, "vt_pad_zero", launch_vt_pad_zero(x.at<bf16_t>(x.w.v), (int64_t)x.B * c.n_kv_heads * c.head_dim, x.S, x.st));
    if (tokens)
        LAUNCH(x, "embed", launch_embed(tokens, x.wt(x.m->plan.emb), x.at<float>(x.w.x), x.T, c.d_model, c.vocab, x.S,
                                        x.P, c.mask_id, x.at<int32_t>(x.w.counters) + CNT_INVALID, x.st));
    return DLM_OK;
}

// Final norm of the draft rows, LM head with fused softmax partials, merge.
dlm_status run_head(Ctx& x, int32_t* top1, float* conf, float* maxlogit, float* logits_out) {
    const dlm_config& c = x.c;
    bf16_t* hfin = x.at<bf16_t>(x.w.hfin);
    LAUNCH(x, "rmsnorm_final", launch_rmsnorm_draft_rows(x.at<float>(x.w.x), x.wt(x.m->plan.gf), hfin, x.B,
                                                         x.S, x.P, x.D, c.d_model, c.norm_eps, x.st));
    GemmArgs a = gemm_args(x.wt(x.m->plan.lm), c.d_model, hfin, c.d_model, c.vocab, x.R, c.d_model);
    a.partials = x.at<float4>(x.w.partials);
    a.group_m = 4;
    a.variant = 12;                                     // ping-pong, third stage for the streamed vocabulary rows (A)
    TRY(gemm(x, "gemm_lm_head", a, EPI_LMHEAD, false, kHeadBM, kHeadBN, 0));
    LAUNCH(x, "lmhead_merge", launch_lmhead_merge(a.partials, x.w.n_vtiles, x.R, top1, conf, maxlogit, x.st));
    if (logits_out) {
        GemmArgs b = gemm_args(x.wt(x.m->plan.lm), c.d_model, hfin, c.d_model, c.vocab, x.R, c.d_model);
        b.out = logits_out;
        b.ldo = c.vocab;
        TRY(gemm(x, "gemm_logits_debug", b, EPI_F32_T, false, 256, 256, 0));
    }
    return DLM_OK;
}

dlm_status check_common(dlm_model* m, int B, int P, int D, void* ws, size_t ws_bytes, Workspace* w) {
    if (!m) return fail(DLM_ERR_INVALID_ARG, "model handle is NULL");
    std::string e = check_shape(B, P, D);
    if (e.empty()) e = check_offsets(m->cfg, (int64_t)B * (P + D));
    if (!e.empty()) return fail(DLM_ERR_INVALID_ARG, e);
    *w = plan_workspace(m->cfg, B, P, D);
    if (!ws) return fail(DLM_ERR_INVALID_ARG, "workspace is NULL");
    if (ws_bytes < w->total)
        return fail(DLM_ERR_WORKSPACE, "workspace too small: need " + std::to_string(w->total) + " bytes, got " +
                                           std::to_string(ws_bytes));
    if (((uintptr_t)ws) % kAlign) return fail(DLM_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
    return DLM_OK;
}

Ctx ctx_for(dlm_model* m, int B, int P, int D, void* ws, const Workspace& w, void* stream) {
    Ctx x{m, m->cfg, (char*)ws, w, (hipStream_t)stream, B, P, D, P + D, B * (P + D), B * D};
    return x;
}

dlm_status step_impl(Ctx& x, int32_t* tokens, const dlm_edit_rule& rule, int32_t* top1_out, float* conf_out,
                     dlm_stats* stats_out, int32_t* eos_out = nullptr) {
    const dlm_config& c = x.c;
    int32_t* counters = x.at<int32_t>(x.w.counters);
    int32_t* eos = counters + CNT_EOS;
    LAUNCH(x, "zero", launch_zero_i32(counters, CNT_WORDS, x.st));
    TRY(run_prologue(x, tokens));
    x.draft_rows_last_ffn = true;
    for (int l = 0; l < c.n_layers; ++l) TRY(run_layer(x, l));
    TRY(run_head(x, x.at<int32_t>(x.w.top1), x.at<float>(x.w.conf), x.at<float>(x.w.maxlogit), nullptr));
    LAUNCH(x, "edit", launch_edit(tokens, x.B, x.S, x.P, x.D, x.at<int32_t>(x.w.top1), x.at<float>(x.w.conf),
                                  rule.unmask_threshold, rule.edit_threshold, c.mask_id, rule.eos_id, counters,
                                  rule.eos_id >= 0 ? eos : nullptr, top1_out, conf_out, x.st));
    if (stats_out) HIP_TRY(hipMemcpyAsync(stats_out, counters, sizeof(dlm_stats), hipMemcpyDeviceToDevice, x.st));
    if (eos_out) HIP_TRY(hipMemcpyAsync(eos_out, eos, 4, hipMemcpyDeviceToDevice, x.st));
    return DLM_OK;
}

// ------------------------------------------------------------ block-AR drafting
// Workspace of drafting (B, P, D, block): window buffers for max(P, block)
// rows per sequence, then the per-layer K / V^T caches over all P + D
// positions, the RoPE table of those positions, the window's tokens and the
// token state [B][P + D].
struct DraftPlan {
    Workspace w;
    size_t kc = 0, vc = 0, rope = 0, wtok = 0, tokens = 0, total = 0;
    size_t kc_layer = 0, vc_layer = 0;
    int rows = 0;
};

DraftPlan plan_draft(const dlm_config& c, int B, int P, int D, int blk) {
    DraftPlan p;
    p.rows = std::max(P, std::min(2 * blk, D));       // a block window may carry the block before it
    p.w = plan_workspace(c, B, 0, p.rows);
    size_t total = p.w.total;
    auto add = [&](int64_t bytes) {
        const size_t off = total;
        total = align_up(total + (size_t)std::max<int64_t>(bytes, 1));
        return off;
    };
    const int64_t S = (int64_t)P + D;
    const int hd = c.head_dim;
    p.kc_layer = (size_t)B * c.n_kv_heads * S * hd;
    p.vc_layer = (size_t)B * c.n_kv_heads * hd * vt_stride((int)S);
    p.kc = add(((int64_t)c.n_layers * p.kc_layer + 64 * hd) * 2);     // + one 64-key tile of tail
    p.vc = add((int64_t)c.n_layers * p.vc_layer * 2);
    p.rope = add(S * (hd / 2) * 8);
    p.wtok = add((int64_t)B * p.rows * 4);
    p.tokens = add((int64_t)B * S * 4);
    p.total = total;
    return p;
}

std::string check_draft_shape(int B, int P, int D, int blk) {
    std::string e = check_shape(B, P, D);
    if (!e.empty()) return e;
    if (blk < 1 || blk > 1024) return "block_len must be in [1, 1024]";
    return "";
}

dlm_status check_draft(dlm_model* m, int B, int P, int D, int blk, void* ws, size_t ws_bytes, DraftPlan* p) {
    if (!m) return fail(DLM_ERR_INVALID_ARG, "model handle is NULL");
    std::string e = check_draft_shape(B, P, D, blk);
    if (e.empty()) e = check_offsets(m->cfg, (int64_t)B * (P + D));
    if (!e.empty()) return fail(DLM_ERR_INVALID_ARG, e);
    *p = plan_draft(m->cfg, B, P, D, blk);
    if (!ws) return fail(DLM_ERR_INVALID_ARG, "workspace is NULL");
    if (ws_bytes < p->total)
        return fail(DLM_ERR_WORKSPACE, "workspace too small: need " + std::to_string(p->total) + " bytes, got " +
                                           std::to_string(ws_bytes));
    if (((uintptr_t)ws) % kAlign) return fail(DLM_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
    return DLM_OK;
}

struct Drafter {
    dlm_model* m;
    char* ws;
    const DraftPlan& p;
    hipStream_t st;
    int B, P, D, S, blk;

    // Context of the window of L rows starting at position c0 of every sequence.
    Ctx window(int c0, int L) const {
        Ctx x{m, m->cfg, ws, p.w, st, B, 0, L, L, B * L, B * L};
        x.q0 = c0;
        x.kv_seq = S;
        x.kc = x.at<bf16_t>(p.kc);
        x.vc = x.at<bf16_t>(p.vc);
        x.kc_layer = p.kc_layer;
        x.vc_layer = p.vc_layer;
        x.rope_all = x.at<float2>(p.rope);
        return x;
    }
    int32_t* counters() const { return reinterpret_cast<int32_t*>(ws + p.w.counters); }

    // Forward of one window of the token state: all layers' K/V of its rows go
    // into the caches; with head, also the top-1 / confidence of its rows from
    // row `lead` on.  The first `lead` rows are a finished block carried along
    // to commit its K/V: they see keys only up to their own end.
    dlm_status run(const int32_t* tokens, int c0, int L, bool head, int lead = 0) const {
        Ctx x = window(c0, L);
        const dlm_config& c = m->cfg;
        x.kv_only = !head;
        if (lead) {
            x.P = lead;
            x.D = L - lead;
            x.R = B * (L - lead);
            x.att_split = lead;
            x.att_keys_lo = c0 + lead;
        }
        int32_t* wtok = x.at<int32_t>(p.wtok);
        LAUNCH(x, "window_gather", launch_window_gather(tokens, wtok, B, S, c0, L, st));
        // a window inside the prompt must hold no [MASK] id; every id must lie in [0, vocab)
        LAUNCH(x, "embed", launch_embed(wtok, x.wt(m->plan.emb), x.at<float>(p.w.x), x.T, c.d_model, c.vocab, L,
                                        c0 + L <= P ? L : 0, c.mask_id, counters() + CNT_INVALID, st));
        for (int l = 0; l < c.n_layers; ++l) TRY(run_layer(x, l));
        if (head) TRY(run_head(x, x.at<int32_t>(p.w.top1), x.at<float>(p.w.conf), x.at<float>(p.w.maxlogit), nullptr));
        HIP_TRY(hipGetLastError());
        return DLM_OK;
    }

    // Fresh caches (zero, so the attention's tile reads past the visible keys
    // meet finite values), the RoPE table, and the prompt's K/V: the prompt
    // attends to itself only.
    dlm_status begin(const int32_t* tokens) const {
        const dlm_config& c = m->cfg;
        Ctx x = window(0, 1);
        launch_fill_bf16(x.kc, (uint64_t)c.n_layers * p.kc_layer + 64 * c.head_dim, 0, st);
        launch_fill_bf16(x.vc, (uint64_t)c.n_layers * p.vc_layer, 0, st);
        launch_rope_table(x.at<float2>(p.rope), S, c.head_dim / 2, (double)c.rope_theta, S, 0, st);
        HIP_TRY(hipGetLastError());
        if (P > 0) TRY(run(tokens, 0, P, false));
        return DLM_OK;
    }

    int block_start(int k) const { return P + k * blk; }
    int block_rows(int k) const { return std::min(blk, S - block_start(k)); }

    // One denoising step on block k: forward of the block's window, then the
    // unmasking.  With with_prev, the window also carries block k-1 (finished,
    // its K/V not yet in the caches), which commits it in the same pass.
    // counters: [0] unmasked, [2] masked left in the block, [3] = 1.
    dlm_status step(int32_t* tokens, int k, float tau, int steps_left, int32_t* top1_out, float* conf_out,
                    bool with_prev = false) const {
        const int c0 = block_start(k), L = block_rows(k);
        if (with_prev)
            TRY(run(tokens, c0 - blk, blk + L, true, blk));
        else
            TRY(run(tokens, c0, L, true));
        Ctx x = window(c0, L);
        launch_zero_i32(counters(), 4, st);
        prof_begin(x, "draft_select");
        hipError_t e = launch_draft_select(tokens, B, S, c0, L, x.at<int32_t>(p.w.top1), x.at<float>(p.w.conf), tau,
                                           steps_left, m->cfg.mask_id, counters(), top1_out, conf_out, st);
        prof_end(x, "draft_select");
        if (e != hipSuccess) return fail(DLM_ERR_HIP, std::string("draft_select: ") + hipGetErrorString(e));
        return DLM_OK;
    }
};

dlm_status fail_invalid_tokens(int n) {
    return fail(DLM_ERR_INVALID_ARG, std::to_string(n) + " token id(s) outside [0, vocab) or [MASK] id(s) in the "
                                     "prompt; the pass wrote nothing");
}

dlm_status check_rule(const dlm_config& c, const dlm_edit_rule* rule) {
    if (!rule) return fail(DLM_ERR_INVALID_ARG, "rule is NULL");
    if (isnan(rule->unmask_threshold) || isnan(rule->edit_threshold)) return fail(DLM_ERR_INVALID_ARG, "threshold is NaN");
    if (rule->eos_id >= c.vocab) return fail(DLM_ERR_INVALID_ARG, "eos_id >= vocab");
    return DLM_OK;
}

}  // namespace

// Workspace of dlm_refine_step_static: a device array of fixed size, one copy
// per GPU for the life of the process.  Host code never passes its name to a
// kernel or a copy (on the host it names a stand-in, not device memory); it
// uses the per-device address that hipGetSymbolAddress returns.
static __device__ __align__(256) char scratch[DLM_STATIC_SCRATCH_BYTES];

namespace {

std::mutex g_scratch_mu;
constexpr int kMaxDevices = 64;
char* g_scratch_ptr[kMaxDevices] = {};

// Address of this process's scratch array on the current device, resolved
// once per device.
dlm_status scratch_on_current_device(char** out, int* dev_out) {
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) return fail(DLM_ERR_UNSUPPORTED, "device index >= 64");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(DLM_ERR_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
        g_scratch_ptr[dev] = static_cast<char*>(p);
    }
    *out = g_scratch_ptr[dev];
    *dev_out = dev;
    return DLM_OK;
}

}  // namespace

extern "C" {

const char* dlm_last_error(void) { return g_last_error.c_str(); }

size_t dlm_weights_bytes(const dlm_config* cfg) {
    try {
        if (!validate(cfg).empty()) return 0;
        return plan_weights(*cfg).total;
    } catch (...) {
        caught_exception();
        return 0;
    }
}

size_t dlm_workspace_bytes(const dlm_config* cfg, int32_t batch, int32_t prompt_len, int32_t draft_len) {
    try {
        if (!validate(cfg).empty() || !check_shape(batch, prompt_len, draft_len).empty()) return 0;
        if (!check_offsets(*cfg, (int64_t)batch * (prompt_len + draft_len)).empty()) return 0;
        return plan_workspace(*cfg, batch, prompt_len, draft_len).total;
    } catch (...) {
        caught_exception();
        return 0;
    }
}

dlm_status dlm_load_synthetic_weights(const dlm_config* cfg, uint64_t seed, void* d_weights,
                                      size_t weights_bytes, void* hip_stream, dlm_model** out) {
    try {
        const std::string e = validate(cfg);
        if (!e.empty()) return fail(DLM_ERR_INVALID_ARG, e);
        if (!out) return fail(DLM_ERR_INVALID_ARG, "out is NULL");
        *out = nullptr;
        if (!d_weights) return fail(DLM_ERR_INVALID_ARG, "weights buffer is NULL");
        if (((uintptr_t)d_weights) % kAlign) return fail(DLM_ERR_INVALID_ARG, "weights buffer must be 256-byte aligned");
        WeightPlan plan = plan_weights(*cfg);
        if (weights_bytes < plan.total)
            return fail(DLM_ERR_WORKSPACE, "weights buffer too small: need " + std::to_string(plan.total) + " bytes");
        char* scratch_ptr = nullptr;
        int dev = 0;
        TRY(scratch_on_current_device(&scratch_ptr, &dev));     // set-up: once per device
        hipStream_t st = (hipStream_t)hip_stream;
        char* base = (char*)d_weights;
        for (const TensorInit& t : plan.inits) {
            bf16_t* dst = reinterpret_cast<bf16_t*>(base + t.off);
            if (t.kind_fill) {
                launch_fill_bf16(dst, t.n_phys, (bf16_t)0x3f80, st);
            } else {
                const float c = (float)((double)cfg->init_std * (double)t.scale * sqrt(3.0) / 65536.0);
                launch_init_weights(dst, t.n_phys, t.cols, t.tid_a, t.tid_b, t.layout, seed, c, st);
            }
            HIP_TRY(hipGetLastError());
        }
        alloc_point();
        dlm_model* m = new dlm_model();
        m->cfg = *cfg;
        m->seed = seed;
        m->device = dev;
        m->scratch = scratch_ptr;
        m->base = base;
        m->bytes = weights_bytes;
        m->plan = std::move(plan);
        *out = m;
        return DLM_OK;
    } catch (...) {
        return caught_exception();
    }
}

dlm_status dlm_refine_step_ex(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t draft_len,
                              int32_t* d_tokens, const dlm_edit_rule* rule, void* d_workspace,
                              size_t workspace_bytes, void* hip_stream, int32_t* d_top1, float* d_conf,
                              dlm_stats* d_stats, int32_t* d_eos_written) {
    try {
        Workspace w;
        TRY(check_common(m, batch, prompt_len, draft_len, d_workspace, workspace_bytes, &w));
        if (!d_tokens) return fail(DLM_ERR_INVALID_ARG, "tokens is NULL");
        TRY(check_rule(m->cfg, rule));
        Ctx x = ctx_for(m, batch, prompt_len, draft_len, d_workspace, w, hip_stream);
        return step_impl(x, d_tokens, *rule, d_top1, d_conf, d_stats, d_eos_written);
    } catch (...) {
        return caught_exception();
    }
}

dlm_status dlm_refine_step(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t draft_len,
                           int32_t* d_tokens, float threshold, void* d_workspace, size_t workspace_bytes,
                           void* hip_stream, int32_t* d_top1, float* d_conf, dlm_stats* d_stats) {
    try {
        const dlm_edit_rule rule{threshold, threshold, -1};
        return dlm_refine_step_ex(m, batch, prompt_len, draft_len, d_tokens, &rule, d_workspace, workspace_bytes,
                                  hip_stream, d_top1, d_conf, d_stats, nullptr);
    } catch (...) {
        return caught_exception();
    }
}

dlm_status dlm_refine_step_static(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t draft_len,
                                  int32_t* d_tokens, float threshold, void* hip_stream, int32_t* d_top1,
                                  float* d_conf, dlm_stats* d_stats) {
    try {
        if (!m) return fail(DLM_ERR_INVALID_ARG, "model handle is NULL");
        std::string e = check_shape(batch, prompt_len, draft_len);
        if (e.empty()) e = check_offsets(m->cfg, (int64_t)batch * (prompt_len + draft_len));
        if (!e.empty()) return fail(DLM_ERR_INVALID_ARG, e);
        if (!d_tokens) return fail(DLM_ERR_INVALID_ARG, "tokens is NULL");
        if (isnan(threshold)) return fail(DLM_ERR_INVALID_ARG, "threshold is NaN");
        int dev = -1;
        HIP_TRY(hipGetDevice(&dev));
        if (dev != m->device || !m->scratch)
            return fail(DLM_ERR_INVALID_ARG, "the model's device (current when its weights were loaded) must be current");
        const Workspace w = plan_workspace(m->cfg, batch, prompt_len, draft_len);
        if (w.total > (size_t)DLM_STATIC_SCRATCH_BYTES)
            return fail(DLM_ERR_WORKSPACE, "this shape needs " + std::to_string(w.total) +
                                               " bytes of workspace; the static scratch holds " +
                                               std::to_string((size_t)DLM_STATIC_SCRATCH_BYTES));
        // Every buffer the pass reads before writing it in the same pass (the
        // counters, the V^T padding) is cleared by a kernel of the pass itself,
        // so whatever an earlier call left in the scratch does not matter.
        const dlm_edit_rule rule{threshold, threshold, -1};
        Ctx x = ctx_for(m, batch, prompt_len, draft_len, m->scratch, w, hip_stream);
        x.no_events = true;
        return step_impl(x, d_tokens, rule, d_top1, d_conf, d_stats, nullptr);
    } catch (...) {
        return caught_exception();
    }
}

dlm_status dlm_refine_ex(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t draft_len,
                         const int32_t* d_prompt, int32_t* d_draft, const uint8_t* d_mask, int32_t n_steps,
                         const dlm_edit_rule* rule, void* d_workspace, size_t workspace_bytes,
                         void* hip_stream, dlm_stats* h_stats, int32_t* h_stop_reason) {
    try {
        Workspace w;
        TRY(check_common(m, batch, prompt_len, draft_len, d_workspace, workspace_bytes, &w));
        if (!d_draft || (prompt_len > 0 && !d_prompt)) return fail(DLM_ERR_INVALID_ARG, "prompt/draft is NULL");
        if (n_steps < 0) return fail(DLM_ERR_INVALID_ARG, "n_steps < 0");
        TRY(check_rule(m->cfg, rule));
        Ctx x = ctx_for(m, batch, prompt_len, draft_len, d_workspace, w, hip_stream);
        int32_t* tokens = x.at<int32_t>(w.tokens);
        int32_t* counters = x.at<int32_t>(w.counters);
        launch_apply_mask(d_prompt, d_draft, d_mask, tokens, batch, prompt_len, draft_len, m->cfg.mask_id, x.st);
        HIP_TRY(hipGetLastError());
        dlm_stats tot{0, 0, 0, 0, 0};
        int32_t reason = 0;
        for (int s = 0; s < n_steps; ++s) {
            TRY(step_impl(x, tokens, *rule, nullptr, nullptr, nullptr));
            int32_t st[CNT_WORDS] = {};                   // the pass counters
            HIP_TRY(hipMemcpyAsync(st, counters, sizeof(st), hipMemcpyDeviceToHost, x.st));
            HIP_TRY(hipStreamSynchronize(x.st));
            if (st[CNT_INVALID]) return fail_invalid_tokens(st[CNT_INVALID]);
            tot.n_unmasked += st[CNT_UNMASKED];
            tot.n_edited += st[CNT_EDITED];
            tot.steps_run += 1;
            if (st[CNT_UNMASKED] + st[CNT_EDITED] == 0) {
                reason = 1;
                break;
            }
            if (rule->eos_id >= 0 && st[CNT_EOS] > 0) {
                reason = 2;
                break;
            }
        }
        launch_copy_draft_out(tokens, d_draft, batch, x.S, prompt_len, draft_len, x.st);
        launch_zero_i32(counters, 4, x.st);
        launch_count_masks(tokens, batch, x.S, prompt_len, draft_len, m->cfg.mask_id, counters + 2, x.st);
        HIP_TRY(hipGetLastError());
        dlm_stats st{};
        HIP_TRY(hipMemcpyAsync(&st, counters, sizeof(st), hipMemcpyDeviceToHost, x.st));
        HIP_TRY(hipStreamSynchronize(x.st));
        tot.n_masked_left = st.n_masked_left;
        if (h_stats) *h_stats = tot;
        if (h_stop_reason) *h_stop_reason = reason;
        return DLM_OK;
    } catch (...) {
        return caught_exception();
    }
}

dlm_status dlm_refine_step_span(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t span_len,
                                int32_t span_start, int32_t* d_tokens, const dlm_edit_rule* rule, void* d_workspace,
                                size_t workspace_bytes, void* hip_stream, int32_t* d_top1, float* d_conf,
                                dlm_stats* d_stats, int32_t* d_eos_written) {
    try {
        Workspace w;
        TRY(check_common(m, batch, prompt_len, span_len, d_workspace, workspace_bytes, &w));
        if (!d_tokens) return fail(DLM_ERR_INVALID_ARG, "tokens is NULL");
        if (span_start < 0) return fail(DLM_ERR_INVALID_ARG, "span_start < 0");
        TRY(check_rule(m->cfg, rule));
        Ctx x = ctx_for(m, batch, prompt_len, span_len, d_workspace, w, hip_stream);
        x.pos_shift = span_start;
        return step_impl(x, d_tokens, *rule, d_top1, d_conf, d_stats, d_eos_written);
    } catch (...) {
        return caught_exception();
    }
}

dlm_status dlm_refine_local(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t draft_len,
                            const int32_t* d_prompt, int32_t* d_draft, const uint8_t* d_mask, int32_t n_stages,
                            const int32_t* h_span, const int32_t* h_passes, const dlm_edit_rule* rule,
                            void* d_workspace, size_t workspace_bytes, void* hip_stream, dlm_stats* h_stats,
                            int32_t* h_stop_reason) {
    try {
        Workspace wfull;
        TRY(check_common(m, batch, prompt_len, draft_len, d_workspace, workspace_bytes, &wfull));
        if (!d_draft || (prompt_len > 0 && !d_prompt)) return fail(DLM_ERR_INVALID_ARG, "prompt/draft is NULL");
        if (n_stages < 0 || (n_stages > 0 && (!h_span || !h_passes))) return fail(DLM_ERR_INVALID_ARG, "bad schedule");
        for (int i = 0; i < n_stages; ++i)
            if (h_span[i] < 1 || h_passes[i] < 0) return fail(DLM_ERR_INVALID_ARG, "span < 1 or passes < 0");
        TRY(check_rule(m->cfg, rule));
        hipStream_t st = (hipStream_t)hip_stream;
        const int n = batch * draft_len;
        if (d_mask) launch_mask_draft(d_draft, d_mask, n, m->cfg.mask_id, st);
        HIP_TRY(hipGetLastError());
        dlm_stats tot{0, 0, 0, 0, 0};
        int32_t reason = 1;                                // every chunk stopped on its own (or nothing ran)
        bool eos_stop = false;
        for (int g = 0; g < n_stages && !eos_stop; ++g) {
            const int L = std::min<int>(h_span[g], draft_len);
            for (int c0 = 0; c0 < draft_len && !eos_stop; c0 += L) {
                const int len = std::min(L, draft_len - c0);
                Workspace w;
                TRY(check_common(m, batch, prompt_len, len, d_workspace, workspace_bytes, &w));
                Ctx x = ctx_for(m, batch, prompt_len, len, d_workspace, w, hip_stream);
                x.pos_shift = c0;
                int32_t* tokens = x.at<int32_t>(w.tokens);
                int32_t* counters = x.at<int32_t>(w.counters);
                launch_span_gather(d_prompt, d_draft, tokens, batch, prompt_len, draft_len, c0, len, st);
                HIP_TRY(hipGetLastError());
                bool still = false;
                for (int p = 0; p < h_passes[g]; ++p) {
                    TRY(step_impl(x, tokens, *rule, nullptr, nullptr, nullptr));
                    int32_t c[CNT_WORDS] = {};
                    HIP_TRY(hipMemcpyAsync(c, counters, sizeof(c), hipMemcpyDeviceToHost, st));
                    HIP_TRY(hipStreamSynchronize(st));
                    if (c[CNT_INVALID]) return fail_invalid_tokens(c[CNT_INVALID]);
                    tot.n_unmasked += c[CNT_UNMASKED];
                    tot.n_edited += c[CNT_EDITED];
                    tot.steps_run += 1;
                    if (c[CNT_UNMASKED] + c[CNT_EDITED] == 0) {
                        still = true;
                        break;
                    }
                    if (rule->eos_id >= 0 && c[CNT_EOS] > 0) {
                        eos_stop = true;
                        break;
                    }
                }
                if (!still && h_passes[g] > 0) reason = reason == 2 ? 2 : 0;
                launch_span_scatter(tokens, d_draft, batch, prompt_len, draft_len, c0, len, st);
                HIP_TRY(hipGetLastError());
            }
        }
        if (eos_stop) reason = 2;
        int32_t* counters = reinterpret_cast<int32_t*>((char*)d_workspace + wfull.counters);
        launch_zero_i32(counters, 4, st);
        launch_count_masks(d_draft, batch, draft_len, 0, draft_len, m->cfg.mask_id, counters + 2, st);
        HIP_TRY(hipGetLastError());
        dlm_stats fin{};
        HIP_TRY(hipMemcpyAsync(&fin, counters, sizeof(fin), hipMemcpyDeviceToHost, st));
        HIP_TRY(hipStreamSynchronize(st));
        tot.n_masked_left = fin.n_masked_left;
        if (h_stats) *h_stats = tot;
        if (h_stop_reason) *h_stop_reason = reason;
        return DLM_OK;
    } catch (...) {
        return caught_exception();
    }
}

dlm_status dlm_refine(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t draft_len,
                      const int32_t* d_prompt, int32_t* d_draft, const uint8_t* d_mask, int32_t n_steps,
                      float threshold, void* d_workspace, size_t workspace_bytes, void* hip_stream,
                      dlm_stats* h_stats) {
    try {
        const dlm_edit_rule rule{threshold, threshold, -1};
        return dlm_refine_ex(m, batch, prompt_len, draft_len, d_prompt, d_draft, d_mask, n_steps, &rule, d_workspace,
                             workspace_bytes, hip_stream, h_stats, nullptr);
    } catch (...) {
        return caught_exception();
    }
}

size_t dlm_draft_workspace_bytes(const dlm_config* cfg, int32_t batch, int32_t prompt_len, int32_t draft_len,
                                 int32_t block_len) {
    try {
        if (!validate(cfg).empty() || !check_draft_shape(batch, prompt_len, draft_len, block_len).empty()) return 0;
        if (!check_offsets(*cfg, (int64_t)batch * (prompt_len + draft_len)).empty()) return 0;
        return plan_draft(*cfg, batch, prompt_len, draft_len, block_len).total;
    } catch (...) {
        caught_exception();
        return 0;
    }
}

dlm_status dlm_draft_step(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t draft_len, int32_t block_len,
                          int32_t block_index, int32_t steps_left, float threshold, int32_t* d_tokens,
                          void* d_workspace, size_t workspace_bytes, void* hip_stream, int32_t* d_top1,
                          float* d_conf, float* d_max_logit, dlm_stats* d_stats) {
    try {
        DraftPlan p;
        TRY(check_draft(m, batch, prompt_len, draft_len, block_len, d_workspace, workspace_bytes, &p));
        if (!d_tokens) return fail(DLM_ERR_INVALID_ARG, "tokens is NULL");
        const int n_blocks = (draft_len + block_len - 1) / block_len;
        if (block_index < 0 || block_index >= n_blocks) return fail(DLM_ERR_INVALID_ARG, "block_index out of range");
        if (steps_left < 1) return fail(DLM_ERR_INVALID_ARG, "steps_left < 1");
        if (isnan(threshold)) return fail(DLM_ERR_INVALID_ARG, "threshold is NaN");
        const Drafter dr{m, (char*)d_workspace, p, (hipStream_t)hip_stream, batch, prompt_len, draft_len,
                         prompt_len + draft_len, block_len};
        launch_zero_i32(dr.counters(), CNT_WORDS, dr.st);
        TRY(dr.begin(d_tokens));
        for (int j = 0; j < block_index; ++j) TRY(dr.run(d_tokens, dr.block_start(j), block_len, false));
        TRY(dr.step(d_tokens, block_index, threshold, steps_left, d_top1, d_conf));
        if (d_stats) HIP_TRY(hipMemcpyAsync(d_stats, dr.counters(), sizeof(dlm_stats), hipMemcpyDeviceToDevice, dr.st));
        if (d_max_logit)
            HIP_TRY(hipMemcpyAsync(d_max_logit, dr.ws + p.w.maxlogit, (size_t)batch * dr.block_rows(block_index) * 4,
                                   hipMemcpyDeviceToDevice, dr.st));
        return DLM_OK;
    } catch (...) {
        return caught_exception();
    }
}

dlm_status dlm_draft(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t draft_len, const int32_t* d_prompt,
                     int32_t* d_draft, int32_t block_len, int32_t steps_per_block, float threshold,
                     void* d_workspace, size_t workspace_bytes, void* hip_stream, dlm_stats* h_stats,
                     int32_t* h_block_steps) {
    try {
        DraftPlan p;
        TRY(check_draft(m, batch, prompt_len, draft_len, block_len, d_workspace, workspace_bytes, &p));
        if (!d_draft || (prompt_len > 0 && !d_prompt)) return fail(DLM_ERR_INVALID_ARG, "prompt/draft is NULL");
        if (steps_per_block < 1) return fail(DLM_ERR_INVALID_ARG, "steps_per_block < 1");
        if (isnan(threshold)) return fail(DLM_ERR_INVALID_ARG, "threshold is NaN");
        const int S = prompt_len + draft_len;
        const Drafter dr{m, (char*)d_workspace, p, (hipStream_t)hip_stream, batch, prompt_len, draft_len, S, block_len};
        int32_t* tokens = reinterpret_cast<int32_t*>((char*)d_workspace + p.tokens);
        launch_zero_i32(dr.counters(), CNT_WORDS, dr.st);
        launch_draft_init(d_prompt, tokens, batch, prompt_len, S, m->cfg.vocab, m->cfg.mask_id, dr.counters(), dr.st);
        HIP_TRY(hipGetLastError());
        TRY(dr.begin(tokens));
        const int n_blocks = (draft_len + block_len - 1) / block_len;
        dlm_stats tot{0, 0, 0, 0, 0};
        for (int k = 0; k < n_blocks; ++k) {
            int used = 0;
            for (int t = 0; t < steps_per_block; ++t) {
                // the first step of a block also commits the previous block's K/V
                TRY(dr.step(tokens, k, threshold, steps_per_block - t, nullptr, nullptr, t == 0 && k > 0));
                int32_t c[CNT_WORDS] = {};
                HIP_TRY(hipMemcpyAsync(c, dr.counters(), sizeof(c), hipMemcpyDeviceToHost, dr.st));
                HIP_TRY(hipStreamSynchronize(dr.st));
                if (c[CNT_INVALID]) return fail_invalid_tokens(c[CNT_INVALID]);
                ++used;
                tot.n_unmasked += c[0];
                if (c[2] == 0) break;                     // no [MASK] left in the block
            }
            tot.steps_run += used;
            if (h_block_steps) h_block_steps[k] = used;
        }
        launch_copy_draft_out(tokens, d_draft, batch, S, prompt_len, draft_len, dr.st);
        launch_zero_i32(dr.counters(), 4, dr.st);
        launch_count_masks(tokens, batch, S, prompt_len, draft_len, m->cfg.mask_id, dr.counters() + 2, dr.st);
        HIP_TRY(hipGetLastError());
        dlm_stats fin{};
        HIP_TRY(hipMemcpyAsync(&fin, dr.counters(), sizeof(fin), hipMemcpyDeviceToHost, dr.st));
        HIP_TRY(hipStreamSynchronize(dr.st));
        tot.n_masked_left = fin.n_masked_left;
        if (h_stats) *h_stats = tot;
        return DLM_OK;
    } catch (...) {
        return caught_exception();
    }
}

size_t dlm_cascade_workspace_bytes(const dlm_config* drafter_cfg, const dlm_config* refiner_cfg, int32_t batch,
                                   int32_t prompt_len, int32_t draft_len, int32_t block_len) {
    try {
        const size_t a = dlm_draft_workspace_bytes(drafter_cfg, batch, prompt_len, draft_len, block_len);
        const size_t b = dlm_workspace_bytes(refiner_cfg, batch, prompt_len, draft_len);
        return a && b ? std::max(a, b) : 0;
    } catch (...) {
        caught_exception();
        return 0;
    }
}

dlm_status dlm_cascade(dlm_model* drafter, dlm_model* refiner, int32_t batch, int32_t prompt_len, int32_t draft_len,
                       const int32_t* d_prompt, int32_t* d_draft, int32_t block_len, int32_t steps_per_block,
                       float draft_threshold, int32_t n_refine_steps, const dlm_edit_rule* rule, void* d_workspace,
                       size_t workspace_bytes, void* hip_stream, dlm_cascade_stats* h_stats) {
    try {
        if (!drafter || !refiner) return fail(DLM_ERR_INVALID_ARG, "model handle is NULL");
        if (drafter->cfg.vocab != refiner->cfg.vocab || drafter->cfg.mask_id != refiner->cfg.mask_id)
            return fail(DLM_ERR_INVALID_ARG, "drafter and refiner must share the vocabulary and the mask id");
        if (n_refine_steps < 0) return fail(DLM_ERR_INVALID_ARG, "n_refine_steps < 0");
        TRY(check_rule(refiner->cfg, rule));
        if (workspace_bytes < dlm_cascade_workspace_bytes(&drafter->cfg, &refiner->cfg, batch, prompt_len, draft_len,
                                                          block_len))
            return fail(DLM_ERR_WORKSPACE, "workspace too small for the cascade");
        using clk = std::chrono::steady_clock;
        dlm_cascade_stats cs{};
        const auto t0 = clk::now();
        TRY(dlm_draft(drafter, batch, prompt_len, draft_len, d_prompt, d_draft, block_len, steps_per_block,
                      draft_threshold, d_workspace, workspace_bytes, hip_stream, &cs.draft, nullptr));
        const auto t1 = clk::now();              // dlm_draft returns with the draft written
        TRY(dlm_refine_ex(refiner, batch, prompt_len, draft_len, d_prompt, d_draft, nullptr, n_refine_steps, rule,
                          d_workspace, workspace_bytes, hip_stream, &cs.refine, &cs.refine_stop_reason));
        const auto t2 = clk::now();              // and so does dlm_refine_ex
        cs.draft_passes = cs.draft.steps_run;
        cs.refine_passes = cs.refine.steps_run;
        cs.draft_ms = std::chrono::duration<double, std::milli>(t1 - t0).count();
        cs.refine_ms = std::chrono::duration<double, std::milli>(t2 - t1).count();
        if (h_stats) *h_stats = cs;
        return DLM_OK;
    } catch (...) {
        return caught_exception();
    }
}

dlm_status dlm_debug_forward(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t draft_len,
                             const int32_t* d_tokens, void* d_workspace, size_t workspace_bytes,
                             void* hip_stream, float* d_hidden, float* d_max_logit, int32_t* d_top1,
                             float* d_conf, float* d_logits, int32_t* d_route_ids, float* d_router_logits) {
    try {
        Workspace w;
        TRY(check_common(m, batch, prompt_len, draft_len, d_workspace, workspace_bytes, &w));
        if (!d_tokens) return fail(DLM_ERR_INVALID_ARG, "tokens is NULL");
        Ctx x = ctx_for(m, batch, prompt_len, draft_len, d_workspace, w, hip_stream);
        TRY(run_prologue(x, d_tokens));
        const size_t route_words = (size_t)x.T * m->cfg.top_k;
        for (int l = 0; l < m->cfg.n_layers; ++l) {
            if (d_router_logits && m->cfg.n_experts > 0)
                x.dbg_router_logits = d_router_logits + (size_t)l * x.T * m->cfg.n_experts;
            TRY(run_layer(x, l));
            if (d_route_ids && m->cfg.n_experts > 0)
                HIP_TRY(hipMemcpyAsync(d_route_ids + l * route_words, x.at<int32_t>(w.ids), route_words * 4,
                                       hipMemcpyDeviceToDevice, x.st));
        }
        if (d_hidden)
            HIP_TRY(hipMemcpyAsync(d_hidden, x.at<float>(w.x), (size_t)x.T * m->cfg.d_model * 4,
                                   hipMemcpyDeviceToDevice, x.st));
        if (d_max_logit || d_top1 || d_conf || d_logits) {
            TRY(run_head(x, x.at<int32_t>(w.top1), x.at<float>(w.conf), x.at<float>(w.maxlogit), d_logits));
            const size_t R = (size_t)x.R;
            if (d_max_logit) HIP_TRY(hipMemcpyAsync(d_max_logit, x.at<float>(w.maxlogit), R * 4, hipMemcpyDeviceToDevice, x.st));
            if (d_top1) HIP_TRY(hipMemcpyAsync(d_top1, x.at<int32_t>(w.top1), R * 4, hipMemcpyDeviceToDevice, x.st));
            if (d_conf) HIP_TRY(hipMemcpyAsync(d_conf, x.at<float>(w.conf), R * 4, hipMemcpyDeviceToDevice, x.st));
        }
        return DLM_OK;
    } catch (...) {
        return caught_exception();
    }
}

dlm_status dlm_debug_layer(dlm_model* m, int32_t layer, int32_t batch, int32_t seq_len, const float* d_x_in,
                           float* d_x_out, void* d_workspace, size_t workspace_bytes, void* hip_stream,
                           int32_t* d_route_ids, float* d_router_logits) {
    try {
        Workspace w;
        TRY(check_common(m, batch, 0, seq_len, d_workspace, workspace_bytes, &w));
        if (layer < 0 || layer >= m->cfg.n_layers) return fail(DLM_ERR_INVALID_ARG, "layer out of range");
        if (!d_x_in || !d_x_out) return fail(DLM_ERR_INVALID_ARG, "x is NULL");
        Ctx x = ctx_for(m, batch, 0, seq_len, d_workspace, w, hip_stream);
        if (m->cfg.n_experts > 0) x.dbg_router_logits = d_router_logits;
        const size_t bytes = (size_t)x.T * m->cfg.d_model * 4;
        HIP_TRY(hipMemcpyAsync(x.at<float>(w.x), d_x_in, bytes, hipMemcpyDeviceToDevice, x.st));
        TRY(run_prologue(x, nullptr));
        TRY(run_layer(x, layer));
        HIP_TRY(hipMemcpyAsync(d_x_out, x.at<float>(w.x), bytes, hipMemcpyDeviceToDevice, x.st));
        if (d_route_ids && m->cfg.n_experts > 0)
            HIP_TRY(hipMemcpyAsync(d_route_ids, x.at<int32_t>(w.ids), (size_t)x.T * m->cfg.top_k * 4,
                                   hipMemcpyDeviceToDevice, x.st));
        return DLM_OK;
    } catch (...) {
        return caught_exception();
    }
}

dlm_status dlm_debug_head(dlm_model* m, int32_t batch, int32_t prompt_len, int32_t draft_len, const float* d_x,
                          void* d_workspace, size_t workspace_bytes, void* hip_stream, float* d_max_logit,
                          int32_t* d_top1, float* d_conf) {
    try {
        Workspace w;
        TRY(check_common(m, batch, prompt_len, draft_len, d_workspace, workspace_bytes, &w));
        if (!d_x) return fail(DLM_ERR_INVALID_ARG, "x is NULL");
        Ctx x = ctx_for(m, batch, prompt_len, draft_len, d_workspace, w, hip_stream);
        HIP_TRY(hipMemcpyAsync(x.at<float>(w.x), d_x, (size_t)x.T * m->cfg.d_model * 4, hipMemcpyDeviceToDevice, x.st));
        TRY(run_head(x, x.at<int32_t>(w.top1), x.at<float>(w.conf), x.at<float>(w.maxlogit), nullptr));
        const size_t R = (size_t)x.R;
        if (d_max_logit) HIP_TRY(hipMemcpyAsync(d_max_logit, x.at<float>(w.maxlogit), R * 4, hipMemcpyDeviceToDevice, x.st));
        if (d_top1) HIP_TRY(hipMemcpyAsync(d_top1, x.at<int32_t>(w.top1), R * 4, hipMemcpyDeviceToDevice, x.st));
        if (d_conf) HIP_TRY(hipMemcpyAsync(d_conf, x.at<float>(w.conf), R * 4, hipMemcpyDeviceToDevice, x.st));
        return DLM_OK;
    } catch (...) {
        return caught_exception();
    }
}

dlm_status dlm_debug_gemm(const void* d_a, const void* d_b, float* d_c, int32_t m, int32_t n, int32_t k,
                          int32_t tile_m, int32_t tile_n, void* hip_stream) {
    try {
        if (!d_a || !d_b || !d_c) return fail(DLM_ERR_INVALID_ARG, "NULL argument");
        if (m <= 0 || n <= 0 || k <= 0 || k % 64) return fail(DLM_ERR_INVALID_ARG, "bad GEMM shape");
        GemmArgs a = gemm_args((const bf16_t*)d_a, k, (const bf16_t*)d_b, k, m, n, k);
        a.out = d_c;
        a.ldo = n;
        a.variant = tile_m >> 16;
        hipError_t e = launch_gemm(a, EPI_F32, false, tile_m & 0xffff, tile_n, 0, (hipStream_t)hip_stream);
        if (e != hipSuccess) return fail(DLM_ERR_INVALID_ARG, std::string("gemm: ") + hipGetErrorString(e));
        return DLM_OK;
    } catch (...) {
        return caught_exception();
    }
}

dlm_status dlm_weight_info(dlm_model* m, int32_t layer_field, int32_t kind, int32_t expert, void** d_ptr,
                           int32_t* layout) {
    try {
        if (!m || !d_ptr || !layout) return fail(DLM_ERR_INVALID_ARG, "NULL argument");
        const dlm_config& c = m->cfg;
        const size_t d = c.d_model;
        if (layer_field == 0) {
            if (kind == 0) { *d_ptr = m->base + m->plan.emb; *layout = 0; return DLM_OK; }
            if (kind == 1) { *d_ptr = m->base + m->plan.lm; *layout = 0; return DLM_OK; }
            return fail(DLM_ERR_INVALID_ARG, "unknown global tensor kind");
        }
        const int l = layer_field - 1;
        if (l < 0 || l >= c.n_layers) return fail(DLM_ERR_INVALID_ARG, "layer out of range");
        const LayerPtrs& L = m->plan.layers[l];
        const size_t nq = (size_t)c.n_heads * c.head_dim, nk = (size_t)c.n_kv_heads * c.head_dim;
        char* b = m->base;
        *layout = 0;
        switch (kind) {
            case K_WQ: *d_ptr = b + L.wqkv; return DLM_OK;
            case K_WK: *d_ptr = b + L.wqkv + nq * d * 2; return DLM_OK;
            case K_WV: *d_ptr = b + L.wqkv + (nq + nk) * d * 2; return DLM_OK;
            case K_WO: *d_ptr = b + L.wo; return DLM_OK;
            default: break;
        }
        if (c.n_experts == 0) {
            if (kind == K_FG || kind == K_FU) { *d_ptr = b + L.wgu; *layout = 1; return DLM_OK; }
            if (kind == K_FD) { *d_ptr = b + L.wd; return DLM_OK; }
            return fail(DLM_ERR_INVALID_ARG, "unknown dense-layer tensor kind");
        }
        const size_t F = c.expert_ffn_dim;
        int e = expert;
        if (kind == K_ROUTER) { *d_ptr = b + L.wr; return DLM_OK; }
        if (kind >= K_SG && kind <= K_SD) {
            if (expert < 0 || expert >= c.n_shared_experts) return fail(DLM_ERR_INVALID_ARG, "shared expert out of range");
            e = c.n_experts + expert;
            kind -= 3;
        } else if (expert < 0 || expert >= c.n_experts) {
            return fail(DLM_ERR_INVALID_ARG, "expert out of range");
        }
        if (kind == K_EG || kind == K_EU) { *d_ptr = b + L.wgu + (size_t)e * 2 * F * d * 2; *layout = 1; return DLM_OK; }
        if (kind == K_ED) { *d_ptr = b + L.wd + (size_t)e * d * F * 2; return DLM_OK; }
        return fail(DLM_ERR_INVALID_ARG, "unknown tensor kind");
    } catch (...) {
        return caught_exception();
    }
}

dlm_status dlm_set_profiling(dlm_model* m, const char* name_filter) {
    try {
        if (!m) return fail(DLM_ERR_INVALID_ARG, "model handle is NULL");
        m->prof_on = name_filter != nullptr;
        m->prof_filter = name_filter ? name_filter : "";
        m->prof_used = 0;
        return DLM_OK;
    } catch (...) {
        return caught_exception();
    }
}

int32_t dlm_profile_read(dlm_model* m, const char** names, float* ms, int32_t max_entries) {
    try {
        if (!m) return -1;
        int32_t n = 0;
        for (size_t i = 0; i < m->prof_used && n < max_entries; ++i) {
            float t = 0.f;
            if (hipEventSynchronize(m->prof[i].b) != hipSuccess) return -1;
            if (hipEventElapsedTime(&t, m->prof[i].a, m->prof[i].b) != hipSuccess) return -1;
            if (names) names[n] = m->prof[i].name;
            if (ms) ms[n] = t;
            ++n;
        }
        return n;
    } catch (...) {
        caught_exception();
        return -1;
    }
}

dlm_status dlm_debug_fail_host_alloc(int32_t n) {
    if (n < 0) return fail(DLM_ERR_INVALID_ARG, "n must be >= 0");
    g_fail_alloc_in.store(n, std::memory_order_relaxed);
    return DLM_OK;
}

void dlm_free(dlm_model* m) {
    if (!m) return;
    for (ProfRec& r : m->prof) {
        if (r.a) hipEventDestroy(r.a);
        if (r.b) hipEventDestroy(r.b);
    }
    delete m;
}

}  // extern "C"
