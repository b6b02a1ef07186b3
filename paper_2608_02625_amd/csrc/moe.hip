// Mixture-of-experts routing for the refiner's FFN: router logits with
// softmax top-k, dispatch (per-expert row ranges + device tile table for the
// grouped GEMM) and the weighted combine back into the residual stream.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace {

// XOR key of the 16-byte chunks of an LDS row of CPR chunks (8, 16 or 32):
// a fragment read of 32 consecutive rows at one logical chunk hits distinct
// banks (with 16 or more chunks per row the low four row bits suffice).
template <int CPR>
__device__ __forceinline__ int rkey(int row) {
    if constexpr (CPR >= 16) return row & 15;
    else return (row & 7) ^ ((row >> 3) & 1);
}

// Router + top-k for 32 tokens per workgroup (8 waves).
// z^T[e][t] = sum_c Wr[e][c] h[t][c] on v_mfma_f32_32x32x16_bf16 with experts
// as rows (NB <= 8 blocks of 32) and tokens as columns.  K advances ROWB / 2
// columns at a time (64, 128 or 256) through 3 to 8 LDS stages that the
// waves fill with buffer loads straight from global memory (whole ROWB-byte
// row segments, 16-byte chunks XOR-swizzled), so every byte of h and Wr is
// fetched once per workgroup in full cache lines.  Each expert block's
// 16-wide K steps are dealt round-robin to 8 / NB waves and the parts are
// added in a fixed order.
// Each wave then selects for 4 tokens; lane r < k records selection r with its
// rank among this workgroup's selections of the same expert (LDS counter), and
// the workgroup's per-expert counts go to wg_counts[E][workgroup].  Ranks only
// order rows inside an expert's group.
template <int NB, int ROWB>
__global__ __launch_bounds__(512) void router_topk_kernel(const bf16_t* __restrict__ h, const bf16_t* __restrict__ Wr,
                                                         int T, int d, int E, int k, int32_t* __restrict__ ids,
                                                         float* __restrict__ wts, int32_t* __restrict__ pos,
                                                         int32_t* __restrict__ wg_counts, float* __restrict__ logits) {
    constexpr int NW = 8;                            // waves
    static_assert(NB >= 1 && NB <= NW, "expert blocks");
    constexpr int KSPLIT = NW / NB;                  // waves sharing an expert block
    constexpr int EP = NB * 32;                      // padded expert count (LDS row)
    constexpr int ZROW = EP + 4;                     // row stride: 16-byte aligned, 4 banks of skew
    constexpr int CPR = ROWB / 16;                   // 16-byte chunks per LDS row
    constexpr int RPB = 1024 / ROWB;                 // rows per 1 KB copy block
    constexpr int HB = 32 / RPB;                     // copy blocks of token rows
    constexpr int KSTEPS = ROWB / 32;                // 16-wide K steps per chunk
    constexpr int H_BYTES = 32 * ROWB, STAGE = H_BYTES + EP * ROWB;
    // Stages: as many as fit in 150 KB (3 to 8), so that several K chunks
    // are in flight while one is multiplied (the K loop is latency-bound).
    constexpr int NS = 150 * 1024 / STAGE < 3 ? 3 : (150 * 1024 / STAGE > 8 ? 8 : 150 * 1024 / STAGE);
    constexpr int NBLK = STAGE / 1024;               // 1 KB copy blocks per stage (RPB rows each)
    constexpr int NI = (NBLK + NW - 1) / NW;         // copies per wave and stage (the last block repeats)
    constexpr int ZBYTES = KSPLIT * 32 * ZROW * 4 + 32 * EP * 8;
    constexpr int LBYTES = NS * STAGE > ZBYTES ? NS * STAGE : ZBYTES;
    __shared__ __attribute__((aligned(16))) char smem[LBYTES];   // K stages, then logit parts and keys
    __shared__ int lcnt[EP];
    typedef float zrow_t[32][ZROW];
    zrow_t* zs = reinterpret_cast<zrow_t*>(smem);
    uint64_t* keys = reinterpret_cast<uint64_t*>(smem + KSPLIT * 32 * ZROW * 4);   // [32][EP]

    // The wave index is made scalar so that branches on it are real
    // branches: an MFMA under an EXEC mask still accumulates.
    const int lane = threadIdx.x & 63, wave = uniform(threadIdx.x >> 6);
    const int g = lane >> 5, j = lane & 31;
    const int t0 = blockIdx.x * 32;
    const int blk0 = wave / KSPLIT, kc = wave % KSPLIT;
    for (int e = threadIdx.x; e < EP; e += NW * 64) lcnt[e] = 0;

    // Copy block q of a stage: q < HB holds token rows RPB q .. RPB q + RPB - 1
    // of h, the others expert rows of Wr (rows past T or E repeat the last one).
    const buf_rsrc_t h_rsrc = make_rsrc(h), w_rsrc = make_rsrc(Wr);
    uint32_t off[NI];
    bool is_h[NI];
    int dst[NI];
#pragma unroll
    for (int p = 0; p < NI; ++p) {
        const int q = min(wave * NI + p, NBLK - 1);
        const int rr = lane / CPR, pc = lane % CPR;
        is_h[p] = q < HB;
        const int row = is_h[p] ? q * RPB + rr : (q - HB) * RPB + rr;
        const int64_t grow = is_h[p] ? min(t0 + row, T - 1) : min(row, E - 1);
        off[p] = (uint32_t)(grow * d * 2) + (uint32_t)((pc ^ rkey<CPR>(row)) * 16);
        dst[p] = q * 1024;
    }
    const lds_ptr_t lds = (lds_ptr_t)smem;
    typedef __attribute__((address_space(3))) char lds_char;
    typedef __attribute__((address_space(3))) const bf16x8 lds_frag;
    auto issue = [&](int c, int stage) {             // K chunk c (ROWB / 2 columns) into a stage
#pragma unroll
        for (int p = 0; p < NI; ++p)
            lds_dma16_buf(is_h[p] ? h_rsrc : w_rsrc, off[p], c * ROWB, (lds_ptr_t)((lds_char*)lds + stage * STAGE + dst[p]));
    };

    f32x16 acc;
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = 0.f;
    const int nk = d / (ROWB / 2);
    const int hfrag = j * ROWB, wfrag = H_BYTES + (blk0 * 32 + j) * ROWB, key = rkey<CPR>(j);
#pragma unroll
    for (int s = 0; s < NS; ++s) issue(min(s, nk - 1), s);
    for (int c = 0; c < nk; ++c) {
        // own copies of K chunk c landed (later chunks may fly), then
        // everyone's; the stage of chunk c-1 is free for chunk c+NS-1
        if (c == 0) wait_vmcnt<NI * (NS - 1)>();
        else wait_vmcnt<NI * (NS - 2)>();
        __syncthreads();
        if (c > 0) issue(min(c + NS - 1, nk - 1), (c + NS - 1) % NS);
        const int sb = (c % NS) * STAGE;
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks) {
            if ((c * KSTEPS + ks) % KSPLIT != kc) continue;   // wave-uniform
            const int co = ((2 * ks + g) ^ key) << 4;
            const bf16x8 wf = *(lds_frag*)((lds_char*)lds + sb + wfrag + co);
            const bf16x8 hf = *(lds_frag*)((lds_char*)lds + sb + hfrag + co);
            acc = mfma32x32x16(wf, hf, acc);
        }
    }
    wait_all_memory();                               // no copy may land in the logit parts
    __syncthreads();
    // acc[e]: expert blk0*32 + 8*(e/4) + 4*g + e%4, token j
#pragma unroll
    for (int e = 0; e < 16; ++e) zs[kc][j][blk0 * 32 + 8 * (e >> 2) + 4 * g + (e & 3)] = acc[e];
    __syncthreads();
    // Sum the K parts in a fixed order; logits of experts >= E become -inf,
    // and so does a NaN logit, so that the order below stays total and every
    // token receives exactly k distinct experts whatever its input.  Each
    // (token, expert) also gets a 64-bit key: the logit's bits made orderable
    // as an unsigned integer above the complement of the expert id, so that
    // "larger logit, or equal logit and lower id" is one unsigned compare.
    for (int i = threadIdx.x; i < 32 * EP; i += NW * 64) {
        const int tt = i / EP, e = i - tt * EP;
        float z = zs[0][tt][e];
#pragma unroll
        for (int s = 1; s < KSPLIT; ++s) z += zs[s][tt][e];
        if (logits && e < E && t0 + tt < T) logits[(int64_t)(t0 + tt) * E + e] = z;   // test hook
        z = (e < E && z == z) ? z + 0.f : -INFINITY;         // (+0.f: -0 and +0 compare equal)
        zs[0][tt][e] = z;
        const uint32_t u = __float_as_uint(z);
        const uint32_t ord = u ^ ((u >> 31) ? 0xffffffffu : 0x80000000u);
        keys[tt * EP + e] = ((uint64_t)ord << 32) | (uint32_t)~e;
    }
    __syncthreads();

    // Top-k per token, four tokens per wave; lane owns experts
    // lane + 64q.  p = softmax(z) over the E experts; expert e is selection
    // r = #{e' : key[e'] > key[e]} if r < k (the k largest logits, ties ->
    // lower id, in descending order); the selected probabilities are
    // renormalised to sum to one.
    constexpr int NQ = (EP + 63) / 64;
    constexpr int TPW = 32 / NW;                     // tokens per wave
    // Ranks of all of the wave's tokens in one pass over the keys (their LDS
    // broadcast reads overlap).
    uint64_t kq[TPW][NQ];
    int rank[TPW][NQ];
#pragma unroll
    for (int i = 0; i < TPW; ++i)
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int e = lane + 64 * q;
            kq[i][q] = e < EP ? keys[(wave * TPW + i) * EP + e] : 0;
            rank[i][q] = 0;
        }
#pragma unroll 8
    for (int e2 = 0; e2 < EP; e2 += 2) {
#pragma unroll
        for (int i = 0; i < TPW; ++i) {
            const uint64_t* kr = keys + (wave * TPW + i) * EP;
            const uint64_t k0 = kr[e2], k1 = kr[e2 + 1];
#pragma unroll
            for (int q = 0; q < NQ; ++q) rank[i][q] += (k0 > kq[i][q]) + (k1 > kq[i][q]);
        }
    }
    for (int i = 0; i < TPW; ++i) {
        const int tt = wave * TPW + i, t = t0 + tt;
        const float* z = zs[0][tt];
        float v[NQ];
        float vm = -INFINITY;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int e = lane + 64 * q;
            v[q] = e < E ? z[e] : -INFINITY;
            vm = fmaxf(vm, v[q]);
        }
        const float m = wave_max_dpp(vm);
        float p[NQ], own = 0.f;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            p[q] = (lane + 64 * q < E) ? __expf(v[q] - m) : 0.f;
            own += p[q];
        }
        const float sum = wave_sum_dpp(own);
        float psel = 0.f;
#pragma unroll
        for (int q = 0; q < NQ; ++q)
            if (rank[i][q] < k) psel += p[q] / sum;
        const float psum = wave_sum_dpp(psel);
        if (t < T) {
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                const int e = lane + 64 * q;
                if (e < E && rank[i][q] < k) {
                    const int64_t o = (int64_t)t * k + rank[i][q];
                    ids[o] = e;
                    wts[o] = p[q] / sum / psum;
                    pos[o] = atomicAdd(&lcnt[e], 1);
                }
            }
        }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += NW * 64) wg_counts[(int64_t)e * gridDim.x + blockIdx.x] = lcnt[e];
}

// Exclusive scan of n <= 512 non-negative ints held in LDS, by one wave;
// out[n] receives the total.
__device__ void wave_scan512(const int* in, int* out, int n) {
    const int lane = threadIdx.x & 63;
    int v[8], run = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int idx = lane * 8 + i;
        v[i] = idx < n ? in[idx] : 0;
        run += v[i];
    }
    int incl = run;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int o = __shfl_up(incl, off, 64);
        if (lane >= off) incl += o;
    }
    int excl = incl - run;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int idx = lane * 8 + i;
        if (idx < n) out[idx] = excl;
        excl += v[i];
    }
    if (lane == 63) out[n] = incl;
}

// Dispatch plan (one workgroup of 16 waves).  The per-workgroup counts of
// each routed expert e, wg_counts[e][0 .. nwg), become exclusive offsets over
// the router workgroups (in place) and their total the group size: 16 threads
// share an expert row, each summing a contiguous segment (loads issued eight
// at a time), then a 16-lane scan gives each segment its start.  Groups are
// the E routed experts followed by n_shared shared experts of T rows each;
// their sizes are scanned into grp_off[0..G], and the tile table (group, m0)
// of the grouped GEMM and its length are written.
__global__ __launch_bounds__(1024) void dispatch_plan_kernel(int T, int E, int n_shared, int nwg, int bm,
                                                             int32_t* __restrict__ wg_counts,
                                                             int32_t* __restrict__ grp_off, int2* __restrict__ tile_tab,
                                                             int32_t* __restrict__ n_tiles) {
    __shared__ int cnt[512], off[513], ntl[512], toff[513];
    const int G = E + n_shared;
    const int wave = threadIdx.x >> 6, sub = threadIdx.x & 15, row = threadIdx.x >> 4;
    const int seg = (nwg + 15) >> 4;
    const int w0 = min(sub * seg, nwg), w1 = min(w0 + seg, nwg);
    for (int e0 = 0; e0 < E; e0 += 64) {
        const int e = e0 + row;
        const bool live = e < E;
        int32_t* col = wg_counts + (int64_t)(live ? e : 0) * nwg;
        int s = 0;
        if (live) {
            for (int w = w0; w < w1; w += 8) {
                int v[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) v[u] = w + u < w1 ? col[w + u] : 0;
#pragma unroll
                for (int u = 0; u < 8; ++u) s += v[u];
            }
        }
        int incl = s;
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
            const int u = __shfl_up(incl, o, 16);
            if (sub >= o) incl += u;
        }
        if (live) {
            int run = incl - s;
            for (int w = w0; w < w1; w += 8) {
                int v[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) v[u] = w + u < w1 ? col[w + u] : 0;
#pragma unroll
                for (int u = 0; u < 8; ++u)
                    if (w + u < w1) {
                        col[w + u] = run;
                        run += v[u];
                    }
            }
            if (sub == 15) cnt[e] = incl;
        }
    }
    for (int gi = E + threadIdx.x; gi < G; gi += blockDim.x) cnt[gi] = T;
    __syncthreads();
    for (int gi = threadIdx.x; gi < G; gi += blockDim.x) ntl[gi] = (cnt[gi] + bm - 1) / bm;
    __syncthreads();
    if (wave == 0) wave_scan512(cnt, off, G);
    else if (wave == 1) wave_scan512(ntl, toff, G);
    __syncthreads();
    for (int gi = threadIdx.x; gi <= G; gi += blockDim.x) grp_off[gi] = off[gi];
    if (threadIdx.x == 0) *n_tiles = toff[G];
    for (int gi = threadIdx.x; gi < G; gi += blockDim.x)
        for (int t = 0; t < ntl[gi]; ++t) tile_tab[toff[gi] + t] = make_int2(gi, t * bm);
}

// Fused dispatch for small count tables: one workgroup per router workgroup
// w (its 32 tokens).  Each workgroup derives from the per-expert counts
// wg_counts[E][nwg] what it needs itself: every group's size (all routed
// experts, then n_shared shared experts of T rows) and, per expert, how many
// of that expert's selections come from router workgroups before w (4
// threads per expert row, each summing a contiguous segment).  Workgroup 0
// also writes grp_off, the tile table and its length.  The selections of the
// workgroup's tokens then get their rows as in dispatch_scatter_kernel.  No
// workgroup waits for another; the redundant reads of the count table
// (E * nwg ints per workgroup) are why this is used for small tables only.
__global__ __launch_bounds__(256) void dispatch_fused_kernel(const int32_t* __restrict__ ids, int T, int k, int E,
                                                              int n_shared, int nwg, int bm,
                                                              const int32_t* __restrict__ wg_counts,
                                                              int32_t* __restrict__ grp_off,
                                                              int2* __restrict__ tile_tab,
                                                              int32_t* __restrict__ n_tiles,
                                                              int32_t* __restrict__ slot, int32_t* __restrict__ a_rows) {
    __shared__ int tot[512], before[512], off[513], ntl[512], toff[513];
    const int w = blockIdx.x, G = E + n_shared;
    const int wave = threadIdx.x >> 6, q = threadIdx.x & 3, er = threadIdx.x >> 2;
    const int seg = (nwg + 3) >> 2;
    const int w0 = min(q * seg, nwg), w1 = min(w0 + seg, nwg);
    for (int e0 = 0; e0 < E; e0 += 64) {
        const int e = e0 + er;
        int s_all = 0, s_pre = 0;
        if (e < E) {
            const int32_t* col = wg_counts + (int64_t)e * nwg;
            for (int v0 = w0; v0 < w1; v0 += 8) {
                int c[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) c[u] = v0 + u < w1 ? col[v0 + u] : 0;
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    s_all += c[u];
                    if (v0 + u < w) s_pre += c[u];
                }
            }
        }
        s_all += __shfl_xor(s_all, 1, 64);
        s_all += __shfl_xor(s_all, 2, 64);
        s_pre += __shfl_xor(s_pre, 1, 64);
        s_pre += __shfl_xor(s_pre, 2, 64);
        if (e < E && q == 0) {
            tot[e] = s_all;
            before[e] = s_pre;
        }
    }
    for (int gi = E + threadIdx.x; gi < G; gi += blockDim.x) tot[gi] = T;
    __syncthreads();
    for (int gi = threadIdx.x; gi < G; gi += blockDim.x) ntl[gi] = (tot[gi] + bm - 1) / bm;
    __syncthreads();
    if (wave == 0) wave_scan512(tot, off, G);
    else if (wave == 1) wave_scan512(ntl, toff, G);
    __syncthreads();
    if (w == 0) {
        for (int gi = threadIdx.x; gi <= G; gi += blockDim.x) grp_off[gi] = off[gi];
        if (threadIdx.x == 0) *n_tiles = toff[G];
        for (int gi = threadIdx.x; gi < G; gi += blockDim.x)
            for (int t = 0; t < ntl[gi]; ++t) tile_tab[toff[gi] + t] = make_int2(gi, t * bm);
    }
    const int t0 = w * 32;
    for (int il = threadIdx.x; il < 32 * k; il += blockDim.x) {
        const int t = t0 + il / k;
        if (t < T) {
            const int64_t i = (int64_t)t0 * k + il;
            const int e = ids[i];
            const int sr = off[e] + before[e] + slot[i];
            slot[i] = sr;
            a_rows[sr] = t;
        }
    }
    for (int il = threadIdx.x; il < 32 * n_shared; il += blockDim.x) {
        const int t = t0 + (il & 31), sh = il >> 5;
        if (t < T) a_rows[off[E + sh] + t] = t;
    }
}

// Thread i < T*k turns the rank pos[i] of selection i into its row
// slot[i] = grp_off[e] + (offset of its router workgroup at e) + pos[i]
// (in place) and sets a_rows[slot] = token; the rest fill the shared groups.
__global__ __launch_bounds__(256) void dispatch_scatter_kernel(const int32_t* __restrict__ ids, int T, int k, int E,
                                                               int n_shared, int nwg, const int32_t* __restrict__ wg_off,
                                                               const int32_t* __restrict__ grp_off,
                                                               int32_t* __restrict__ slot, int32_t* __restrict__ a_rows) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    const int nr = T * k;
    if (i < nr) {
        const int t = i / k, e = ids[i];
        const int s = grp_off[e] + wg_off[(int64_t)e * nwg + (t >> 5)] + slot[i];
        slot[i] = s;
        a_rows[s] = t;
    } else if (i < nr + n_shared * T) {
        const int r = i - nr, sh = r / T, t = r - sh * T;
        a_rows[grp_off[E + sh] + t] = t;
    }
}

// x[t] += sum_j w[t][j] * Y[slot[t][j]] + sum_s Y[grp_off[E+s] + t], fixed order.
// With g_next, also the next block's input norm h[t] = bf16(x[t] / rms * g_next)
// (the same arithmetic, in the same order, as the stand-alone RMSNorm).
// NR = k + n_shared rows per token, a compile-time count so that all of a
// token's row loads are issued before the first is used.
template <int NR>
__global__ void combine_kernel(float* __restrict__ x, const bf16_t* __restrict__ Y,
                               const int32_t* __restrict__ slot, const float* __restrict__ w,
                               const int32_t* __restrict__ grp_off, int k, int E, int n_shared,
                               int d, const bf16_t* __restrict__ g_next, bf16_t* __restrict__ h_next, float eps,
                               int map_S, int map_P, int map_D) {
    const int t = blockIdx.x;
    const int64_t xrow = map_D > 0 ? (int64_t)(t / map_D) * map_S + map_P + t % map_D : t;
    int rows[NR];
    float wt[NR];
#pragma unroll
    for (int r = 0; r < NR; ++r) {
        if (r < k) {
            rows[r] = slot[(int64_t)t * k + r];
            wt[r] = w[(int64_t)t * k + r];
        } else {
            rows[r] = grp_off[E + (r - k)] + t;
            wt[r] = 1.f;
        }
    }
    float* xr = x + xrow * d;
    float ss = 0.f;
    for (int i = threadIdx.x * 8; i < d; i += blockDim.x * 8) {
        u32x4 y[NR];
#pragma unroll
        for (int r = 0; r < NR; ++r) y[r] = *reinterpret_cast<const u32x4*>(Y + (int64_t)rows[r] * d + i);
        float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            const float c = wt[r];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                acc[2 * q] += c * __uint_as_float(y[r][q] << 16);
                acc[2 * q + 1] += c * __uint_as_float(y[r][q] & 0xffff0000u);
            }
        }
        f32x4 a = *reinterpret_cast<const f32x4*>(xr + i);
        f32x4 b = *reinterpret_cast<const f32x4*>(xr + i + 4);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            a[q] += acc[q];
            b[q] += acc[q + 4];
        }
        *reinterpret_cast<f32x4*>(xr + i) = a;
        *reinterpret_cast<f32x4*>(xr + i + 4) = b;
        ss += a[0] * a[0] + a[1] * a[1] + a[2] * a[2] + a[3] * a[3];
        ss += b[0] * b[0] + b[1] * b[1] + b[2] * b[2] + b[3] * b[3];
    }
    if (g_next) rms_store_row(xr, g_next, h_next + (int64_t)t * d, d, block_rms_scale(ss, d, eps));
}

template <int NB>
void launch_router_nb(int rowb, dim3 grid, hipStream_t st, const bf16_t* h, const bf16_t* Wr, int T, int d, int E,
                      int k, int32_t* ids, float* w, int32_t* pos, int32_t* wg_counts, float* logits) {
    if constexpr (NB <= 2) {
        if (rowb == 512) {
            hipLaunchKernelGGL((router_topk_kernel<NB, 512>), grid, dim3(512), 0, st, h, Wr, T, d, E, k, ids, w, pos,
                               wg_counts, logits);
            return;
        }
    }
    if constexpr (NB <= 4) {
        if (rowb == 256) {
            hipLaunchKernelGGL((router_topk_kernel<NB, 256>), grid, dim3(512), 0, st, h, Wr, T, d, E, k, ids, w, pos,
                               wg_counts, logits);
            return;
        }
    }
    hipLaunchKernelGGL((router_topk_kernel<NB, 128>), grid, dim3(512), 0, st, h, Wr, T, d, E, k, ids, w, pos,
                       wg_counts, logits);
}

}  // namespace

hipError_t launch_router_topk(const bf16_t* h, const bf16_t* Wr, int T, int d, int E, int k, int32_t* ids,
                              float* w, int32_t* pos, int32_t* wg_counts, hipStream_t st, float* logits) {
    if (E < 1 || E > 256 || k < 1 || k > 8 || k > E || d % 64 != 0 || T < 1) return hipErrorInvalidValue;
    if ((int64_t)T * d * 2 >= ((int64_t)1 << 31)) return hipErrorInvalidValue;   // 32-bit buffer offsets into h
    const dim3 grid((T + 31) / 32), block(512);
    // The widest K chunk (256, 128 or 64 columns: 512, 256 or 128-byte LDS
    // rows, so the fewest stage barriers) that divides d and whose three
    // stages fit in the LDS with the expert rows.
    const int nb = E <= 32 ? 1 : E <= 64 ? 2 : E <= 128 ? 4 : 8;
    const int rowb = nb <= 2 && d % 256 == 0 ? 512 : nb <= 4 && d % 128 == 0 ? 256 : 128;
    if (E <= 32)
        launch_router_nb<1>(rowb, grid, st, h, Wr, T, d, E, k, ids, w, pos, wg_counts, logits);
    else if (E <= 64)
        launch_router_nb<2>(rowb, grid, st, h, Wr, T, d, E, k, ids, w, pos, wg_counts, logits);
    else if (E <= 128)
        launch_router_nb<4>(rowb, grid, st, h, Wr, T, d, E, k, ids, w, pos, wg_counts, logits);
    else
        launch_router_nb<8>(rowb, grid, st, h, Wr, T, d, E, k, ids, w, pos, wg_counts, logits);
    return hipGetLastError();
}

hipError_t launch_dispatch(const int32_t* ids, int T, int k, int E, int n_shared, int bm, int32_t* wg_counts,
                           int32_t* grp_off, int2* tile_tab, int32_t* n_tiles, int32_t* slot, int32_t* a_rows,
                           hipStream_t st) {
    if (E + n_shared > 512) return hipErrorInvalidValue;
    const int nwg = (T + 31) / 32;
    if ((int64_t)E * nwg <= 16384) {
        hipLaunchKernelGGL(dispatch_fused_kernel, dim3(nwg), dim3(256), 0, st, ids, T, k, E, n_shared, nwg, bm,
                           wg_counts, grp_off, tile_tab, n_tiles, slot, a_rows);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(dispatch_plan_kernel, dim3(1), dim3(1024), 0, st, T, E, n_shared, nwg, bm, wg_counts,
                       grp_off, tile_tab, n_tiles);
    const int64_t n = (int64_t)T * k + (int64_t)n_shared * T;
    hipLaunchKernelGGL(dispatch_scatter_kernel, dim3((unsigned)std::max<int64_t>(1, (n + 255) / 256)), dim3(256), 0,
                       st, ids, T, k, E, n_shared, nwg, wg_counts, grp_off, slot, a_rows);
    return hipGetLastError();
}

void launch_combine(float* x, const bf16_t* Y, const int32_t* slot, const float* w,
                    const int32_t* grp_off, int T, int k, int E, int n_shared, int d, const bf16_t* g_next,
                    bf16_t* h_next, float eps, hipStream_t st, int map_S, int map_P, int map_D) {
    const int nr = k + std::min(n_shared, 9 - k);
#define COMBINE_CASE(N)                                                                                    \
    case N:                                                                                                \
        hipLaunchKernelGGL(combine_kernel<N>, dim3(T), dim3(256), 0, st, x, Y, slot, w, grp_off, k, E, n_shared, d, \
                           g_next, h_next, eps, map_S, map_P, map_D);                                      \
        break;
    switch (nr) {
        COMBINE_CASE(1)
        COMBINE_CASE(2)
        COMBINE_CASE(3)
        COMBINE_CASE(4)
        COMBINE_CASE(5)
        COMBINE_CASE(6)
        COMBINE_CASE(7)
        COMBINE_CASE(8)
        COMBINE_CASE(9)
        default:
            break;
    }
#undef COMBINE_CASE
}
