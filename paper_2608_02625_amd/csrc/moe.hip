// Mixture-of-experts routing for the refiner's FFN: softmax router top-k,
// dispatch (per-expert row ranges + device tile table for the grouped GEMM)
// and the weighted combine back into the residual stream.
#include "common.h"
#include "kernels.h"

namespace {

// One wave per token.  p = softmax(z) over all E experts; the k largest
// logits are selected (ties -> lower expert id) and their probabilities are
// renormalised to sum to one.
__global__ void topk_kernel(const float* __restrict__ logits, int T, int E, int k,
                            int32_t* __restrict__ ids, float* __restrict__ w) {
    const int lane = threadIdx.x & 63;
    const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (t >= T) return;
    const float* z = logits + (int64_t)t * E;
    float v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int e = lane + 64 * q;
        v[q] = (e < E) ? z[e] : -INFINITY;
    }
    float m = fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3]));
    m = wave_max(m);
    float sum = 0.f;
#pragma unroll
    for (int q = 0; q < 4; ++q) sum += (lane + 64 * q < E) ? __expf(v[q] - m) : 0.f;
    sum = wave_sum(sum);

    bool sel[4] = {false, false, false, false};
    int isel[8];
    float psel[8];
    float psum = 0.f;
    for (int r = 0; r < k; ++r) {
        float bv = -INFINITY;
        int be = 0x7fffffff;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = lane + 64 * q;
            if (e < E && !sel[q] && (v[q] > bv || be == 0x7fffffff)) {
                bv = v[q];
                be = e;
            }
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            const float ov = __shfl_xor(bv, off, 64);
            const int oe = __shfl_xor(be, off, 64);
            if (ov > bv || (ov == bv && oe < be)) {
                bv = ov;
                be = oe;
            }
        }
        if (be >= E) be = 0;   // only reachable with non-finite logits; keeps ids in range
        if ((be & 63) == lane) sel[be >> 6] = true;
        isel[r] = be;
        psel[r] = __expf(bv - m) / sum;
        psum += psel[r];
    }
    if (lane == 0) {
        for (int r = 0; r < k; ++r) {
            ids[(int64_t)t * k + r] = isel[r];
            w[(int64_t)t * k + r] = psel[r] / psum;
        }
    }
}

// One workgroup (1024 threads) builds the whole dispatch from the top-k ids:
// groups are the E routed experts (rows = tokens routed there) followed by
// n_shared shared experts (T rows each).  Writes grp_off[0..G], the tile table
// (group, m0) of the grouped GEMM and its length, slot[t][j] (the row of
// token t's j-th expert) and a_rows[row] = token.  Histogram and cursors live
// in LDS; the row order inside a group depends on atomic order but no result
// does (rows are computed independently and combined by slot).
__global__ __launch_bounds__(1024) void dispatch_kernel(const int32_t* __restrict__ ids, int T, int k, int E,
                                                        int n_shared, int bm, int32_t* __restrict__ grp_off,
                                                        int2* __restrict__ tile_tab, int32_t* __restrict__ n_tiles,
                                                        int32_t* __restrict__ slot, int32_t* __restrict__ a_rows) {
    __shared__ int cnt[512];
    __shared__ int off[513];
    __shared__ int toff[513];
    const int G = E + n_shared;
    const int nr = T * k;
    for (int g = threadIdx.x; g < G; g += blockDim.x) cnt[g] = (g < E) ? 0 : T;
    __syncthreads();
    for (int i = threadIdx.x; i < nr; i += blockDim.x) atomicAdd(&cnt[ids[i]], 1);
    __syncthreads();
    if (threadIdx.x == 0) {
        int o = 0, to = 0;
        for (int g = 0; g < G; ++g) {
            off[g] = o;
            toff[g] = to;
            o += cnt[g];
            to += (cnt[g] + bm - 1) / bm;
        }
        off[G] = o;
        toff[G] = to;
        *n_tiles = to;
        grp_off[G] = o;
    }
    __syncthreads();
    for (int g = threadIdx.x; g < G; g += blockDim.x) {
        grp_off[g] = off[g];
        const int nt = toff[g + 1] - toff[g];
        for (int t = 0; t < nt; ++t) tile_tab[toff[g] + t] = make_int2(g, t * bm);
        cnt[g] = 0;                                   // reused as the per-group cursor
    }
    __syncthreads();
    for (int i = threadIdx.x; i < nr; i += blockDim.x) {
        const int e = ids[i];
        const int s = off[e] + atomicAdd(&cnt[e], 1);
        slot[i] = s;
        a_rows[s] = i / k;
    }
    for (int i = threadIdx.x; i < n_shared * T; i += blockDim.x) {
        const int sh = i / T, t = i - sh * T;
        a_rows[off[E + sh] + t] = t;
    }
}

// x[t] += sum_j w[t][j] * Y[slot[t][j]] + sum_s Y[grp_off[E+s] + t], fixed order.
__global__ void combine_kernel(float* __restrict__ x, const bf16_t* __restrict__ Y,
                               const int32_t* __restrict__ slot, const float* __restrict__ w,
                               const int32_t* __restrict__ grp_off, int k, int E, int n_shared,
                               int d) {
    const int t = blockIdx.x;
    int rows[9];
    float wt[9];
    int nrow = 0;
    for (int j = 0; j < k; ++j) {
        rows[nrow] = slot[(int64_t)t * k + j];
        wt[nrow++] = w[(int64_t)t * k + j];
    }
    for (int s = 0; s < n_shared && nrow < 9; ++s) {
        rows[nrow] = grp_off[E + s] + t;
        wt[nrow++] = 1.f;
    }
    float* xr = x + (int64_t)t * d;
    for (int i = threadIdx.x * 8; i < d; i += blockDim.x * 8) {
        float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        for (int r = 0; r < nrow; ++r) {
            const u32x4 y = *reinterpret_cast<const u32x4*>(Y + (int64_t)rows[r] * d + i);
            const float c = wt[r];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                acc[2 * q] += c * __uint_as_float(y[q] << 16);
                acc[2 * q + 1] += c * __uint_as_float(y[q] & 0xffff0000u);
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
    }
}

}  // namespace

void launch_topk(const float* logits, int T, int E, int k, int32_t* ids, float* w, hipStream_t st) {
    hipLaunchKernelGGL(topk_kernel, dim3((T + 3) / 4), dim3(256), 0, st, logits, T, E, k, ids, w);
}

void launch_dispatch(const int32_t* ids, int T, int k, int E, int n_shared, int bm, int32_t* grp_off,
                     int2* tile_tab, int32_t* n_tiles, int32_t* slot, int32_t* a_rows, hipStream_t st) {
    hipLaunchKernelGGL(dispatch_kernel, dim3(1), dim3(1024), 0, st, ids, T, k, E, n_shared, bm, grp_off,
                       tile_tab, n_tiles, slot, a_rows);
}

void launch_combine(float* x, const bf16_t* Y, const int32_t* slot, const float* w,
                    const int32_t* grp_off, int T, int k, int E, int n_shared, int d, hipStream_t st) {
    hipLaunchKernelGGL(combine_kernel, dim3(T), dim3(256), 0, st, x, Y, slot, w, grp_off, k, E,
                       n_shared, d);
}
