// Bandwidth-bound kernels of the refinement pass: embedding gather, RMSNorm,
// merge of the LM-head softmax partials, and the threshold edit/unmask rule.
#include "common.h"
#include "kernels.h"

namespace {

// x[t][:] = E[tok[t]][:] (bf16 -> fp32); one workgroup per token.
// Ids outside [0, V) are clamped into range so that no read leaves the table,
// and counted in *invalid together with [MASK] ids in the first mask_rows
// positions of each row of S tokens (the prompt, which must hold real tokens).
__global__ void embed_kernel(const int32_t* __restrict__ tok, const bf16_t* __restrict__ emb,
                             float* __restrict__ x, int d, int V, int S, int mask_rows, int mask_id,
                             int32_t* __restrict__ invalid) {
    const int t = blockIdx.x;
    const int raw = tok[t];
    if (threadIdx.x == 0 && invalid && (raw < 0 || raw >= V || (t % S < mask_rows && raw == mask_id)))
        atomicAdd(invalid, 1);
    const int id = min(max(raw, 0), V - 1);
    const bf16_t* src = emb + (int64_t)id * d;
    float* dst = x + (int64_t)t * d;
    for (int i = threadIdx.x * 8; i < d; i += blockDim.x * 8) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(src + i);
        f32x4 lo, hi;
#pragma unroll
        for (int w = 0; w < 2; ++w) {
            lo[2 * w] = __uint_as_float(v[w] << 16);
            lo[2 * w + 1] = __uint_as_float(v[w] & 0xffff0000u);
            hi[2 * w] = __uint_as_float(v[w + 2] << 16);
            hi[2 * w + 1] = __uint_as_float(v[w + 2] & 0xffff0000u);
        }
        *reinterpret_cast<f32x4*>(dst + i) = lo;
        *reinterpret_cast<f32x4*>(dst + i + 4) = hi;
    }
}

// h = bf16(x / sqrt(mean(x^2) + eps) * g), fp32 math; one workgroup (256) per row.
__device__ __forceinline__ void rmsnorm_row(const float* __restrict__ xr, const bf16_t* __restrict__ g,
                                            bf16_t* __restrict__ hr, int d, float eps) {
    float ss = 0.f;
    for (int i = threadIdx.x * 8; i < d; i += blockDim.x * 8) {
        const f32x4 a = *reinterpret_cast<const f32x4*>(xr + i);
        const f32x4 b = *reinterpret_cast<const f32x4*>(xr + i + 4);
        ss += a[0] * a[0] + a[1] * a[1] + a[2] * a[2] + a[3] * a[3];
        ss += b[0] * b[0] + b[1] * b[1] + b[2] * b[2] + b[3] * b[3];
    }
    rms_store_row(xr, g, hr, d, block_rms_scale(ss, d, eps));
}

__global__ void rmsnorm_kernel(const float* __restrict__ x, const bf16_t* __restrict__ g,
                               bf16_t* __restrict__ h, int d, float eps) {
    const int64_t r = blockIdx.x;
    rmsnorm_row(x + r * d, g, h + r * d, d, eps);
}

__global__ void rmsnorm_draft_kernel(const float* __restrict__ x, const bf16_t* __restrict__ g,
                                     bf16_t* __restrict__ h, int S, int P, int D, int d, float eps) {
    const int r = blockIdx.x;
    const int b = r / D, i = r - b * D;
    rmsnorm_row(x + ((int64_t)b * S + P + i) * d, g, h + (int64_t)r * d, d, eps);
}

// Merge the per-vocabulary-tile partials of each row.  A workgroup handles 8
// rows; each of the 32 thread groups of a row takes every 32nd tile (online
// merge in tile order; one read covers 8 consecutive rows = 128 contiguous
// bytes), then the 32 group results are merged in group order through LDS.
// The order is fixed, so results are deterministic; ties keep the lower
// vocabulary id.
__global__ __launch_bounds__(256) void lmhead_merge_kernel(const float4* __restrict__ part, int n_tiles, int R,
                                                           int32_t* __restrict__ top1, float* __restrict__ conf,
                                                           float* __restrict__ max_logit) {
    __shared__ float4 red[32][8];
    const int rl = threadIdx.x & 7, split = threadIdx.x >> 3;
    const int r = blockIdx.x * 8 + rl;
    SoftmaxPartial acc{-INFINITY, 0x7fffffff, 0.f};
    if (r < R) {
        for (int t = split; t < n_tiles; t += 32) {
            const float4 p = part[(int64_t)t * R + r];
            acc = sp_merge(acc, SoftmaxPartial{p.x, __float_as_int(p.y), p.z});
        }
    }
    red[split][rl] = make_float4(acc.m, __int_as_float(acc.idx), acc.s, 0.f);
    __syncthreads();
    if (split == 0 && r < R) {
        SoftmaxPartial a = acc;
        for (int q = 1; q < 32; ++q) {
            const float4 p = red[q][rl];
            a = sp_merge(a, SoftmaxPartial{p.x, __float_as_int(p.y), p.z});
        }
        top1[r] = a.idx;
        conf[r] = 1.f / a.s;
        if (max_logit) max_logit[r] = a.m;
    }
}

// Threshold rule, all draft slots at once from the same forward pass.
__global__ void edit_kernel(int32_t* __restrict__ tokens, int S, int P, int D,
                            const int32_t* __restrict__ top1, const float* __restrict__ conf,
                            float thr_unmask, float thr_edit, int mask_id, int eos_id,
                            int32_t* __restrict__ counters, int32_t* __restrict__ eos_count,
                            int32_t* __restrict__ out_top1, float* __restrict__ out_conf, int n) {
    const int r = blockIdx.x * blockDim.x + threadIdx.x;
    int unm = 0, edt = 0, eos = 0;
    const bool rejected = counters[CNT_INVALID] != 0;      // the pass saw invalid token ids
    if (r < n) {
        const int b = r / D, i = r - b * D;
        int32_t* slot = tokens + (int64_t)b * S + P + i;
        const int32_t cur = *slot;
        const int32_t t = top1[r];
        const float c = conf[r];
        const float thr = cur == mask_id ? thr_unmask : thr_edit;
        if (!rejected && t != mask_id && c >= thr && t != cur) {
            *slot = t;
            if (cur == mask_id) unm = 1; else edt = 1;
            eos = t == eos_id;
        }
        if (out_top1) out_top1[r] = t;
        if (out_conf) out_conf[r] = c;
    }
    const unsigned long long bu = __ballot(unm), be = __ballot(edt), bx = __ballot(eos);
    if ((threadIdx.x & 63) == 0) {
        if (bu) atomicAdd(&counters[CNT_UNMASKED], (int)__popcll(bu));
        if (be) atomicAdd(&counters[CNT_EDITED], (int)__popcll(be));
        if (bx && eos_count) atomicAdd(eos_count, (int)__popcll(bx));
    }
}

__global__ void span_gather_kernel(const int32_t* __restrict__ prompt, const int32_t* __restrict__ draft,
                                   int32_t* __restrict__ tokens, int P, int D, int c0, int L, int n) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= n) return;
    const int S = P + L;
    const int b = idx / S, s = idx - b * S;
    tokens[idx] = s < P ? prompt[(int64_t)b * P + s] : draft[(int64_t)b * D + c0 + (s - P)];
}

__global__ void span_scatter_kernel(const int32_t* __restrict__ tokens, int32_t* __restrict__ draft, int P, int D,
                                    int c0, int L, int n) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= n) return;
    const int b = idx / L, i = idx - b * L;
    draft[(int64_t)b * D + c0 + i] = tokens[(int64_t)b * (P + L) + P + i];
}

__global__ void mask_draft_kernel(int32_t* __restrict__ draft, const uint8_t* __restrict__ mask, int n, int mask_id) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx < n && mask[idx]) draft[idx] = mask_id;
}

__global__ void apply_mask_kernel(const int32_t* __restrict__ prompt, const int32_t* __restrict__ draft,
                                  const uint8_t* __restrict__ mask, int32_t* __restrict__ tokens,
                                  int P, int D, int mask_id, int n) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= n) return;
    const int S = P + D;
    const int b = idx / S, s = idx - b * S;
    int32_t v;
    if (s < P) {
        v = prompt[(int64_t)b * P + s];
    } else {
        const int64_t di = (int64_t)b * D + (s - P);
        v = (mask && mask[di]) ? mask_id : draft[di];
    }
    tokens[idx] = v;
}

__global__ void copy_draft_out_kernel(const int32_t* __restrict__ tokens, int32_t* __restrict__ draft,
                                      int S, int P, int D, int n) {
    const int r = blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= n) return;
    const int b = r / D, i = r - b * D;
    draft[r] = tokens[(int64_t)b * S + P + i];
}

__global__ void count_masks_kernel(const int32_t* __restrict__ tokens, int S, int P, int D,
                                   int mask_id, int32_t* __restrict__ counter, int n) {
    const int r = blockIdx.x * blockDim.x + threadIdx.x;
    int hit = 0;
    if (r < n) {
        const int b = r / D, i = r - b * D;
        hit = tokens[(int64_t)b * S + P + i] == mask_id;
    }
    const unsigned long long bm = __ballot(hit);
    if ((threadIdx.x & 63) == 0 && bm) atomicAdd(counter, (int)__popcll(bm));
}

// Block-AR drafting: tokens [B][S] = prompt ‖ all [MASK]; prompt ids outside
// [0, V) or equal to the [MASK] id are counted as invalid.
__global__ void draft_init_kernel(const int32_t* __restrict__ prompt, int32_t* __restrict__ tokens, int P, int S,
                                  int V, int mask_id, int32_t* __restrict__ counters, int n) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    int bad = 0;
    if (idx < n) {
        const int b = idx / S, s = idx - b * S;
        const int32_t v = s < P ? prompt[(int64_t)b * P + s] : mask_id;
        bad = s < P && (v < 0 || v >= V || v == mask_id);
        tokens[idx] = v;
    }
    const unsigned long long bb = __ballot(bad);
    if ((threadIdx.x & 63) == 0 && bb) atomicAdd(&counters[CNT_INVALID], (int)__popcll(bb));
}

// out [B][L] = tokens[b][c0 .. c0 + L) of a [B][S] sequence.
__global__ void window_gather_kernel(const int32_t* __restrict__ tokens, int32_t* __restrict__ out, int S, int c0,
                                     int L, int n) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= n) return;
    const int b = idx / L, i = idx - b * L;
    out[idx] = tokens[(int64_t)b * S + c0 + i];
}

// One drafting step's unmasking on the L slots of a block, one workgroup per
// sequence: quota = ceil(masked / steps_left); every masked slot with conf >=
// tau is taken, or, when those are fewer than the quota, the quota masked
// slots of highest confidence (equal confidences: lower position first).  A
// slot's rank among the masked slots is counted directly (L <= 1024).
// counters[0] += slots that took a real token, counters[2] += masked slots
// left afterwards, counters[3] = 1 (one step; the dlm_stats layout).
__global__ __launch_bounds__(256) void draft_select_kernel(int32_t* __restrict__ tokens, int S, int c0, int L,
                                                           const int32_t* __restrict__ top1,
                                                           const float* __restrict__ conf, float tau,
                                                           int steps_left, int mask_id,
                                                           int32_t* __restrict__ counters,
                                                           int32_t* __restrict__ out_top1,
                                                           float* __restrict__ out_conf) {
    __shared__ float cs[1024];
    __shared__ int ms[1024];
    __shared__ int n_mask, n_above, n_unm, n_left;
    const int b = blockIdx.x;
    if (counters[CNT_INVALID] != 0) return;              // the step saw invalid token ids: no update
    int32_t* row = tokens + (int64_t)b * S + c0;
    if (threadIdx.x == 0) n_mask = n_above = n_unm = n_left = 0;
    __syncthreads();
    for (int i = threadIdx.x; i < L; i += blockDim.x) {
        const float c = conf[(int64_t)b * L + i];
        const int m = row[i] == mask_id;
        cs[i] = c;
        ms[i] = m;
        if (m) {
            atomicAdd(&n_mask, 1);
            if (c >= tau) atomicAdd(&n_above, 1);
        }
        if (out_top1) out_top1[(int64_t)b * L + i] = top1[(int64_t)b * L + i];
        if (out_conf) out_conf[(int64_t)b * L + i] = c;
    }
    __syncthreads();
    const int quota = (n_mask + steps_left - 1) / steps_left;
    const int n_sel = max(quota, n_above);
    for (int i = threadIdx.x; i < L; i += blockDim.x) {
        if (!ms[i]) continue;
        const float c = cs[i];
        int rank = 0;
        for (int j = 0; j < L; ++j) rank += ms[j] && (cs[j] > c || (cs[j] == c && j < i));
        int t = mask_id;
        if (rank < n_sel) {
            t = top1[(int64_t)b * L + i];
            row[i] = t;
        }
        if (t != mask_id) atomicAdd(&n_unm, 1);
        else atomicAdd(&n_left, 1);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        if (n_unm) atomicAdd(&counters[0], n_unm);
        if (n_left) atomicAdd(&counters[2], n_left);
        if (b == 0) counters[3] = 1;
    }
}

__global__ void zero_i32_kernel(int32_t* __restrict__ p, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}


__global__ void vt_pad_zero_kernel(bf16_t* vt, int64_t n, int S, int pad, int stride) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const int64_t r = i / pad;
    vt[r * stride + vt_pos(S + (int)(i - r * pad))] = 0;
}

}  // namespace

void launch_embed(const int32_t* tokens, const bf16_t* emb, float* x, int T, int d, int V, int S, int mask_rows,
                  int mask_id, int32_t* invalid, hipStream_t st) {
    hipLaunchKernelGGL(embed_kernel, dim3(T), dim3(256), 0, st, tokens, emb, x, d, V, S, mask_rows, mask_id, invalid);
}

void launch_rmsnorm(const float* x, const bf16_t* g, bf16_t* h, int rows, int d, float eps,
                    hipStream_t st) {
    hipLaunchKernelGGL(rmsnorm_kernel, dim3(rows), dim3(256), 0, st, x, g, h, d, eps);
}

void launch_rmsnorm_draft_rows(const float* x, const bf16_t* g, bf16_t* h, int B, int S, int P,
                               int D, int d, float eps, hipStream_t st) {
    hipLaunchKernelGGL(rmsnorm_draft_kernel, dim3(B * D), dim3(256), 0, st, x, g, h, S, P, D, d, eps);
}

void launch_lmhead_merge(const float4* partials, int n_tiles, int R, int32_t* top1, float* conf,
                         float* max_logit, hipStream_t st) {
    hipLaunchKernelGGL(lmhead_merge_kernel, dim3((R + 7) / 8), dim3(256), 0, st, partials,
                       n_tiles, R, top1, conf, max_logit);
}

void launch_edit(int32_t* tokens, int B, int S, int P, int D, const int32_t* top1, const float* conf,
                 float thr_unmask, float thr_edit, int mask_id, int eos_id, int32_t* counters, int32_t* eos_count,
                 int32_t* out_top1, float* out_conf, hipStream_t st) {
    const int n = B * D;
    hipLaunchKernelGGL(edit_kernel, dim3((n + 255) / 256), dim3(256), 0, st, tokens, S, P, D, top1,
                       conf, thr_unmask, thr_edit, mask_id, eos_id, counters, eos_count, out_top1, out_conf, n);
}

void launch_span_gather(const int32_t* prompt, const int32_t* draft, int32_t* tokens, int B, int P, int D,
                        int c0, int L, hipStream_t st) {
    const int n = B * (P + L);
    hipLaunchKernelGGL(span_gather_kernel, dim3((n + 255) / 256), dim3(256), 0, st, prompt, draft, tokens, P, D, c0,
                       L, n);
}

void launch_span_scatter(const int32_t* tokens, int32_t* draft, int B, int P, int D, int c0, int L, hipStream_t st) {
    const int n = B * L;
    hipLaunchKernelGGL(span_scatter_kernel, dim3((n + 255) / 256), dim3(256), 0, st, tokens, draft, P, D, c0, L, n);
}

void launch_mask_draft(int32_t* draft, const uint8_t* mask, int n, int mask_id, hipStream_t st) {
    hipLaunchKernelGGL(mask_draft_kernel, dim3((n + 255) / 256), dim3(256), 0, st, draft, mask, n, mask_id);
}

void launch_apply_mask(const int32_t* prompt, const int32_t* draft, const uint8_t* mask,
                       int32_t* tokens, int B, int P, int D, int mask_id, hipStream_t st) {
    const int n = B * (P + D);
    hipLaunchKernelGGL(apply_mask_kernel, dim3((n + 255) / 256), dim3(256), 0, st, prompt, draft,
                       mask, tokens, P, D, mask_id, n);
}

void launch_copy_draft_out(const int32_t* tokens, int32_t* draft, int B, int S, int P, int D,
                           hipStream_t st) {
    const int n = B * D;
    hipLaunchKernelGGL(copy_draft_out_kernel, dim3((n + 255) / 256), dim3(256), 0, st, tokens, draft,
                       S, P, D, n);
}

void launch_count_masks(const int32_t* tokens, int B, int S, int P, int D, int mask_id,
                        int32_t* counter, hipStream_t st) {
    const int n = B * D;
    hipLaunchKernelGGL(count_masks_kernel, dim3((n + 255) / 256), dim3(256), 0, st, tokens, S, P, D,
                       mask_id, counter, n);
}

void launch_draft_init(const int32_t* prompt, int32_t* tokens, int B, int P, int S, int V, int mask_id,
                       int32_t* counters, hipStream_t st) {
    const int n = B * S;
    hipLaunchKernelGGL(draft_init_kernel, dim3((n + 255) / 256), dim3(256), 0, st, prompt, tokens, P, S, V, mask_id,
                       counters, n);
}

void launch_window_gather(const int32_t* tokens, int32_t* out, int B, int S, int c0, int L, hipStream_t st) {
    const int n = B * L;
    hipLaunchKernelGGL(window_gather_kernel, dim3((n + 255) / 256), dim3(256), 0, st, tokens, out, S, c0, L, n);
}

hipError_t launch_draft_select(int32_t* tokens, int B, int S, int c0, int L, const int32_t* top1, const float* conf,
                               float tau, int steps_left, int mask_id, int32_t* counters, int32_t* out_top1,
                               float* out_conf, hipStream_t st) {
    if (L < 1 || L > 1024 || steps_left < 1 || c0 < 0 || c0 + L > S) return hipErrorInvalidValue;
    hipLaunchKernelGGL(draft_select_kernel, dim3(B), dim3(256), 0, st, tokens, S, c0, L, top1, conf, tau, steps_left,
                       mask_id, counters, out_top1, out_conf);
    return hipGetLastError();
}

void launch_zero_i32(int32_t* p, int n, hipStream_t st) {
    hipLaunchKernelGGL(zero_i32_kernel, dim3((n + 255) / 256), dim3(256), 0, st, p, n);
}

void launch_vt_pad_zero(bf16_t* vt, int64_t rows, int S, hipStream_t st) {
    const int stride = vt_stride(S), pad = stride - S;
    const int64_t n = rows * pad;
    if (n == 0) return;
    hipLaunchKernelGGL(vt_pad_zero_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, vt, n, S, pad, stride);
}
