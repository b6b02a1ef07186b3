// Host-side launchers of the refinement-step kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef uint16_t bf16_t;

// ----------------------------------------------------------------- init.hip
void launch_init_weights(bf16_t* dst, uint64_t n_phys, uint32_t cols, uint32_t tid_a,
                         uint32_t tid_b, int layout, uint64_t seed, float c, hipStream_t st);
void launch_fill_bf16(bf16_t* dst, uint64_t n, bf16_t v, hipStream_t st);
// RoPE (cos, sin) table [S][half]; rows >= P take position row + shift.
void launch_rope_table(float2* tab, int S, int half, double theta, int P, int shift, hipStream_t st);

// V is kept transposed for attention: V^T [B][KV][hd][S64], S64 = S rounded up
// to the 64-key attention tile.  Inside each aligned group of 16 keys the keys
// are stored in the order an MFMA fragment consumes them: position of key s =
// s with bits 2 and 3 exchanged (keys 4-7 and 8-11 of the group trade
// places).  Positions of keys >= S are zero.
__host__ __device__ inline int vt_pos(int s) { return (s & ~12) | ((s & 4) << 1) | ((s & 8) >> 1); }
__host__ __device__ inline int vt_stride(int S) { return (S + 63) & ~63; }

// ----------------------------------------------------------------- gemm.hip
enum GemmEpilogue {
    EPI_BF16 = 0,     // out_bf16[row][col]
    EPI_F32 = 1,      // out_f32[row][col]
    EPI_RESID = 2,    // resid_f32[row][col] += acc
    EPI_SWIGLU = 3,   // out_bf16[row][f] = silu(gate) * up, gate/up interleaved in 32-col blocks
    EPI_QKV = 4,      // RoPE on q,k; scatter to Q [B][H][S][hd], K [B][KV][Skv][hd], V^T (vt_pos)
    EPI_LMHEAD = 5,   // rows = vocab, cols = tokens: per-(vocab tile, token) softmax partials
    EPI_F32_T = 6,    // out_f32[col][row] (transposed store)
};

struct GemmArgs {
    // C[M x N] = A[M x K] * B[N x K]^T  (bf16 in, fp32 accumulate)
    const bf16_t* A;
    int64_t lda;
    const bf16_t* B;
    int64_t ldb;
    int64_t b_group_stride;   // elements between consecutive groups' B (grouped mode)
    int M, N, K;
    // grouped mode (experts): tiles listed on the device
    const int2* tile_tab;     // [max_tiles] (group, m0)
    const int* n_tiles;       // device scalar: valid entries in tile_tab
    const int* grp_off;       // [groups+1] row offsets (exclusive scan of group sizes)
    const int* a_rows;        // optional gather: A row of permuted row r (NULL = identity)
    int group_m;              // raster: m-tiles per raster group (dense mode)
    int variant;              // K-pipeline variant (0 default; 1 alternative stage/BK choice)
    // epilogue
    void* out;
    int64_t ldo;
    // EPI_QKV
    bf16_t* q;
    bf16_t* k;
    bf16_t* v;
    const float2* rope;       // [kv_seq][hd/2] (cos, sin), by absolute position
    int seq, n_heads, n_kv, head_dim;
    // K and V^T hold kv_seq rows per sequence; token s of a sequence (s < seq)
    // sits at position pos0 + s there and in the RoPE table (refinement: kv_seq
    // = seq, pos0 = 0).  Q keeps seq rows per sequence.
    int kv_seq, pos0;
    // EPI_LMHEAD: partials [2 * ceil(M/BM) half tiles][N] (m, idx, s) stored as float4
    float4* partials;
};

// Launch one GEMM; bm/bn pick the tile (256x256, 256x128, 128x256, 128x128, 128x64).
// max_tiles (grouped mode): capacity of tile_tab.
hipError_t launch_gemm(const GemmArgs& a, int epi, bool grouped, int bm, int bn, int max_tiles,
                       hipStream_t st);

// ----------------------------------------------------------------- attention.hip
// Non-causal attention over Q [B][H][S][hd], K, V [B][KV][S][hd]; O [B*S][H*hd] bf16.
// Draft windows: Q holds Sq rows per sequence, K and V^T hold Skv rows per
// sequence of which the first n_keys are visible (n_keys <= Skv); O [B*Sq][H*hd].
// With q_split > 0 the first q_split query rows see only the first n_keys_lo
// keys (1 <= n_keys_lo <= n_keys).
hipError_t launch_attention(const bf16_t* q, const bf16_t* k, const bf16_t* v, bf16_t* o, int B,
                            int Sq, int Skv, int n_keys, int H, int KV, int hd, hipStream_t st, int q_split = 0,
                            int n_keys_lo = 0);

// Per-pass counters in the workspace (int32 words; the first five are the
// dlm_stats layout).
enum PassCounter {
    CNT_UNMASKED = 0,     // [MASK] slots that took a token
    CNT_EDITED = 1,       // real-token slots that changed
    CNT_MASKED_LEFT = 2,
    CNT_STEPS = 3,
    CNT_INVALID = 4,      // token ids outside [0, V), or [MASK] ids in the prompt
    CNT_EOS = 5,          // slots newly set to the EOS id
    CNT_WORDS = 6
};

// ----------------------------------------------------------------- elementwise.hip
// x[t] = E[tokens[t]] for T = rows of S tokens.  Ids outside [0, V) are
// clamped for the read and counted in *invalid, as are [MASK] ids among the
// first mask_rows tokens of each row of S (the prompt).
void launch_embed(const int32_t* tokens, const bf16_t* emb, float* x, int T, int d, int V, int S, int mask_rows,
                  int mask_id, int32_t* invalid, hipStream_t st);
void launch_rmsnorm(const float* x, const bf16_t* g, bf16_t* h, int rows, int d, float eps,
                    hipStream_t st);
// rows (b, P + i) for i < D of a [B][S] stream -> h [B*D][d]
void launch_rmsnorm_draft_rows(const float* x, const bf16_t* g, bf16_t* h, int B, int S, int P,
                               int D, int d, float eps, hipStream_t st);
void launch_lmhead_merge(const float4* partials, int n_tiles, int R, int32_t* top1, float* conf,
                         float* max_logit, hipStream_t st);
// Threshold update of every draft slot ([MASK] slots against thr_unmask,
// real tokens against thr_edit); counters[CNT_UNMASKED] += unmasked,
// counters[CNT_EDITED] += edited, *eos_count (if not null) += slots newly set
// to eos_id.  Nothing is written when counters[CNT_INVALID] is set.
void launch_edit(int32_t* tokens, int B, int S, int P, int D, const int32_t* top1, const float* conf,
                 float thr_unmask, float thr_edit, int mask_id, int eos_id, int32_t* counters,
                 int32_t* eos_count, int32_t* out_top1, float* out_conf, hipStream_t st);
void launch_apply_mask(const int32_t* prompt, const int32_t* draft, const uint8_t* mask,
                       int32_t* tokens, int B, int P, int D, int mask_id, hipStream_t st);
// Draft spans refined on their own: tokens [B][P + L] = prompt ‖ draft[:, c0 : c0 + L]
// (draft rows of D), and back; mask_id into the masked slots of the draft.
void launch_span_gather(const int32_t* prompt, const int32_t* draft, int32_t* tokens, int B, int P, int D,
                        int c0, int L, hipStream_t st);
void launch_span_scatter(const int32_t* tokens, int32_t* draft, int B, int P, int D, int c0, int L, hipStream_t st);
void launch_mask_draft(int32_t* draft, const uint8_t* mask, int n, int mask_id, hipStream_t st);
void launch_copy_draft_out(const int32_t* tokens, int32_t* draft, int B, int S, int P, int D,
                           hipStream_t st);
void launch_count_masks(const int32_t* tokens, int B, int S, int P, int D, int mask_id,
                        int32_t* counter, hipStream_t st);
void launch_zero_i32(int32_t* p, int n, hipStream_t st);
// Block-AR drafting: tokens [B][S] = prompt ‖ [MASK] ... (prompt ids outside
// [0, V) or equal to mask_id counted in counters[CNT_INVALID]); out [B][L] =
// tokens[:, c0 : c0 + L]; the unmasking of one step on the block at c0 of
// length L <= 1024 (top1 / conf [B][L]; counters[0] += slots given a real
// token, counters[2] += masked slots left, counters[3] = 1; nothing is
// written when counters[CNT_INVALID] is set).
void launch_draft_init(const int32_t* prompt, int32_t* tokens, int B, int P, int S, int V, int mask_id,
                       int32_t* counters, hipStream_t st);
void launch_window_gather(const int32_t* tokens, int32_t* out, int B, int S, int c0, int L, hipStream_t st);
hipError_t launch_draft_select(int32_t* tokens, int B, int S, int c0, int L, const int32_t* top1, const float* conf,
                               float tau, int steps_left, int mask_id, int32_t* counters, int32_t* out_top1,
                               float* out_conf, hipStream_t st);
// Zero the V^T positions of keys S .. S64-1 in every one of `rows` rows.
void launch_vt_pad_zero(bf16_t* vt, int64_t rows, int S, hipStream_t st);

// ----------------------------------------------------------------- moe.hip
// Router logits of T tokens (h [T][d] bf16, Wr [E][d] bf16, E <= 256), softmax
// top-k (k <= 8; ties -> lower id) with renormalised weights.  Tokens are
// handled 32 per router workgroup: pos[t][j] = rank of the selection among its
// workgroup's selections of expert ids[t][j]; wg_counts[E][ceil(T/32)] = per
// expert and workgroup selection counts.  logits (may be null): the router
// logits float [T][E] (test hook).
hipError_t launch_router_topk(const bf16_t* h, const bf16_t* Wr, int T, int d, int E, int k, int32_t* ids,
                              float* w, int32_t* pos, int32_t* wg_counts, hipStream_t st, float* logits = nullptr);
// Group row ranges (E routed + n_shared groups of T rows), tile table of the
// grouped GEMM (tile height bm), slot[t][j] (from pos, in place) and
// a_rows[row] = token.  wg_counts is turned into per-workgroup offsets.
hipError_t launch_dispatch(const int32_t* ids, int T, int k, int E, int n_shared, int bm, int32_t* wg_counts,
                           int32_t* grp_off, int2* tile_tab, int32_t* n_tiles, int32_t* slot, int32_t* a_rows,
                           hipStream_t st);
// x[t] += sum_j w[t][j] * Y[slot[t][j]] + sum_s Y[shared rows]
// With g_next != nullptr, also writes h_next = RMSNorm(x) * g_next (bf16) for
// the next block (the combine holds each finished residual row).
// With map_D > 0 the T tokens are the draft rows of a [B][map_S] stream:
// token t adds into residual row (t / map_D) * map_S + map_P + t % map_D.
void launch_combine(float* x, const bf16_t* Y, const int32_t* slot, const float* w,
                    const int32_t* grp_off, int T, int k, int E, int n_shared, int d,
                    const bf16_t* g_next, bf16_t* h_next, float eps, hipStream_t st, int map_S = 0,
                    int map_P = 0, int map_D = 0);
