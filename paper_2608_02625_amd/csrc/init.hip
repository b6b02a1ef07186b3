// Synthetic weight generation and small per-pass tables.
//
// Weight element i of logical tensor `tid` (row-major [out][in]) is an
// Irwin-Hall draw from Philox4x32-10 (Salmon et al., SC'11):
//   counter = (i_lo, i_hi, tid, 0), key = (seed_lo, seed_hi)
//   n = lo16(w0) + hi16(w0) + lo16(w1) + hi16(w1) - 131070
//   w = bf16_rne(float(n) * c),  c = float(init_std * scale * sqrt(3) / 65536)
#include "common.h"
#include "kernels.h"

namespace {

__device__ __forceinline__ void philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        const uint32_t lo0 = 0xD2511F53u * c[0];
        const uint32_t hi0 = __umulhi(0xD2511F53u, c[0]);
        const uint32_t lo1 = 0xCD9E8D57u * c[2];
        const uint32_t hi1 = __umulhi(0xCD9E8D57u, c[2]);
        const uint32_t n0 = hi1 ^ c[1] ^ k0;
        const uint32_t n2 = hi0 ^ c[3] ^ k1;
        c[0] = n0;
        c[1] = lo1;
        c[2] = n2;
        c[3] = lo0;
    }
}

__device__ __forceinline__ bf16_t weight_value(uint64_t seed, uint32_t tid, uint64_t i, float c) {
    uint32_t ctr[4] = {(uint32_t)i, (uint32_t)(i >> 32), tid, 0u};
    philox4x32_10(ctr, (uint32_t)seed, (uint32_t)(seed >> 32));
    const int32_t s = (int32_t)(ctr[0] & 0xffffu) + (int32_t)(ctr[0] >> 16) +
                      (int32_t)(ctr[1] & 0xffffu) + (int32_t)(ctr[1] >> 16);
    const float v = __fmul_rn((float)(s - 131070), c);
    return f32_to_bf16(v);
}

// Each thread writes 8 consecutive physical elements (16 bytes).
// layout 0: physical == logical [rows][cols] of tid_a.
// layout 1: physical [2*rows][cols]; physical row p belongs to block p/64;
//           rows 0..31 of a block are tid_a (gate) rows, 32..63 tid_b (up).
__global__ void init_weights_kernel(bf16_t* __restrict__ dst, uint64_t n_phys, uint32_t cols,
                                    uint32_t tid_a, uint32_t tid_b, int layout, uint64_t seed,
                                    float c) {
    const uint64_t base = ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) * 8;
    if (base >= n_phys) return;
    uint32_t packed[4];
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
        bf16_t v[2];
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const uint64_t p = base + e + q;
            uint32_t tid = tid_a;
            uint64_t li = p;
            if (layout == 1) {
                const uint64_t prow = p / cols, col = p % cols;
                const uint64_t blk = prow >> 6, w = prow & 63;
                const uint64_t lrow = blk * 32 + (w & 31);
                tid = (w < 32) ? tid_a : tid_b;
                li = lrow * cols + col;
            }
            v[q] = (p < n_phys) ? weight_value(seed, tid, li, c) : (bf16_t)0;
        }
        packed[e / 2] = (uint32_t)v[0] | ((uint32_t)v[1] << 16);
    }
    if (base + 8 <= n_phys) {
        *reinterpret_cast<u32x4*>(dst + base) = u32x4{packed[0], packed[1], packed[2], packed[3]};
    } else {
        for (int e = 0; e < 8 && base + e < n_phys; ++e)
            dst[base + e] = (bf16_t)(packed[e / 2] >> (16 * (e & 1)));
    }
}

__global__ void fill_bf16_kernel(bf16_t* __restrict__ dst, uint64_t n, bf16_t v) {
    const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) dst[i] = v;
}

// cos/sin table [S][half] for rotate-half RoPE, angle = pos * theta^(-2i/hd),
// evaluated in double and rounded to float.  Row s holds position s for the
// first P rows and s + shift after them (a draft span refined on its own keeps
// its positions in the full sequence).
__global__ void rope_table_kernel(float2* __restrict__ tab, int S, int half, double theta, int P, int shift) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= S * half) return;
    const int row = idx / half, i = idx % half;
    const int pos = row < P ? row : row + shift;
    const double inv = pow(theta, -2.0 * (double)i / (double)(2 * half));
    double s, c;
    sincos((double)pos * inv, &s, &c);
    tab[idx] = make_float2((float)c, (float)s);
}

}  // namespace

void launch_init_weights(bf16_t* dst, uint64_t n_phys, uint32_t cols, uint32_t tid_a,
                         uint32_t tid_b, int layout, uint64_t seed, float c, hipStream_t st) {
    const uint64_t threads = (n_phys + 7) / 8;
    const uint64_t blocks = (threads + 255) / 256;
    hipLaunchKernelGGL(init_weights_kernel, dim3((unsigned)blocks), dim3(256), 0, st, dst, n_phys,
                       cols, tid_a, tid_b, layout, seed, c);
}

void launch_fill_bf16(bf16_t* dst, uint64_t n, bf16_t v, hipStream_t st) {
    hipLaunchKernelGGL(fill_bf16_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, dst, n, v);
}

void launch_rope_table(float2* tab, int S, int half, double theta, int P, int shift, hipStream_t st) {
    const int n = S * half;
    hipLaunchKernelGGL(rope_table_kernel, dim3((n + 255) / 256), dim3(256), 0, st, tab, S, half, theta, P, shift);
}
