// Non-causal (bidirectional) grouped-query attention for the refinement pass.
//
// Every query attends to all S keys of its sequence: the refiner revises any
// draft position using context from the whole prompt+draft (paper Sec. 4.2),
// so there is no causal or block mask.  Keys beyond S (tile padding) are the
// only masked entries.
//
// One workgroup = 4 waves = 128 queries of one (batch, head); each wave owns 32
// queries.  K tiles [64 keys][hd] and V^T tiles [hd][64 keys] are staged in LDS
// (two stages, register-prefetched).  Scores are computed transposed,
// S^T = K Q^T, so that each lane owns one query column: the online-softmax
// statistics stay lane-local (plus one exchange with lane^32), and the
// probabilities feed the next MFMA directly from registers as the B operand of
// O^T = V^T P^T, with the matching key order read from the V^T tile.  V is
// stored row-major like K and transposed while it is written to LDS.
#include "common.h"
#include "kernels.h"

namespace {

template <int HD>
struct AttnCfg {
    static constexpr int KEYS = 64;
    static constexpr int K_STRIDE = HD * 2 + 16;      // bytes per K row in LDS
    static constexpr int V_STRIDE = KEYS * 2 + 8;     // bytes per V^T row in LDS
    static constexpr int K_BYTES = KEYS * K_STRIDE;
    static constexpr int V_BYTES = HD * V_STRIDE;
    static constexpr int STAGE = K_BYTES + V_BYTES;
    static constexpr int K_CHUNKS_ROW = HD / 8;       // 16-byte chunks per K row
    static constexpr int K_PASSES = KEYS * K_CHUNKS_ROW / 256;
    static constexpr int V_PASSES = HD / 8 / 4;       // 16-byte V chunks per lane (lane = key)
    static constexpr int NB = HD / 32;                // 32-row blocks of O^T
    static constexpr int NKS = HD / 16;               // K16 steps over hd
};

template <int HD>
__global__ __launch_bounds__(256) void attn_kernel(const bf16_t* __restrict__ Q,
                                                   const bf16_t* __restrict__ K,
                                                   const bf16_t* __restrict__ V,
                                                   bf16_t* __restrict__ O, int S, int H,
                                                   int KV, float scale_log2) {
    using C = AttnCfg<HD>;
    __shared__ __attribute__((aligned(16))) char smem[2 * C::STAGE];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 5, j = lane & 31;
    const int qb = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const int kvh = h / (H / KV);
    const int q = qb * 128 + wave * 32 + j;

    const bf16_t* Qh = Q + ((int64_t)b * H + h) * S * HD;
    const bf16_t* Kh = K + ((int64_t)b * KV + kvh) * S * HD;
    const bf16_t* Vh = V + ((int64_t)b * KV + kvh) * S * HD;

    bf16x8 qf[C::NKS];
    {
        const bf16_t* qp = Qh + (int64_t)min(q, S - 1) * HD + g * 8;
#pragma unroll
        for (int ks = 0; ks < C::NKS; ++ks) qf[ks] = *reinterpret_cast<const bf16x8*>(qp + ks * 16);
    }

    f32x16 oacc[C::NB];
#pragma unroll
    for (int n = 0; n < C::NB; ++n)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[n][e] = 0.f;
    float m_run = -INFINITY, l_run = 0.f;

    // staging registers
    u32x4 rk[C::K_PASSES], rv[C::V_PASSES];
    const int kc = tid % C::K_CHUNKS_ROW, kr = tid / C::K_CHUNKS_ROW;
    constexpr int K_ROWS_PER_PASS = 256 / C::K_CHUNKS_ROW;

    auto gload = [&](int k0) {
#pragma unroll
        for (int p = 0; p < C::K_PASSES; ++p) {
            const int key = k0 + kr + p * K_ROWS_PER_PASS;
            u32x4 v = *reinterpret_cast<const u32x4*>(Kh + (int64_t)min(key, S - 1) * HD + kc * 8);
            if (key >= S) v = u32x4{0u, 0u, 0u, 0u};
            rk[p] = v;
        }
#pragma unroll
        for (int p = 0; p < C::V_PASSES; ++p) {
            const int key = k0 + lane;
            const int chunk = wave + 4 * p;
            u32x4 v = *reinterpret_cast<const u32x4*>(Vh + (int64_t)min(key, S - 1) * HD + chunk * 8);
            if (key >= S) v = u32x4{0u, 0u, 0u, 0u};
            rv[p] = v;
        }
    };
    auto lstore = [&](int buf) {
        char* Ks = smem + buf * C::STAGE;
        char* Vs = Ks + C::K_BYTES;
#pragma unroll
        for (int p = 0; p < C::K_PASSES; ++p)
            *reinterpret_cast<u32x4*>(Ks + (kr + p * K_ROWS_PER_PASS) * C::K_STRIDE + kc * 16) = rk[p];
#pragma unroll
        for (int p = 0; p < C::V_PASSES; ++p) {
            char* dst = Vs + (wave + 4 * p) * 8 * C::V_STRIDE + lane * 2;
#pragma unroll
            for (int i = 0; i < 8; ++i)
                *reinterpret_cast<bf16_t*>(dst + i * C::V_STRIDE) = (bf16_t)(rv[p][i >> 1] >> (16 * (i & 1)));
        }
    };

    const int nkt = (S + C::KEYS - 1) / C::KEYS;
    gload(0);
    lstore(0);
    __syncthreads();
    for (int kt = 0; kt < nkt; ++kt) {
        if (kt + 1 < nkt) gload((kt + 1) * C::KEYS);
        const char* Ks = smem + (kt & 1) * C::STAGE;
        const char* Vs = Ks + C::K_BYTES;
        const int k0 = kt * C::KEYS;

        // S^T for 64 keys (two 32-key chunks): lane holds query j, keys
        // c*32 + 8*(e/4) + 4*g + e%4.
        f32x16 st[2];
#pragma unroll
        for (int c = 0; c < 2; ++c) {
#pragma unroll
            for (int e = 0; e < 16; ++e) st[c][e] = 0.f;
            const char* krow = Ks + (c * 32 + j) * C::K_STRIDE + g * 16;
#pragma unroll
            for (int ks = 0; ks < C::NKS; ++ks) {
                const bf16x8 kf = *reinterpret_cast<const bf16x8*>(krow + ks * 32);
                st[c] = mfma32x32x16(kf, qf[ks], st[c]);
            }
        }
        float mt = -INFINITY;
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int key = k0 + c * 32 + 8 * (e >> 2) + 4 * g + (e & 3);
                const float s = (key < S) ? st[c][e] * scale_log2 : -INFINITY;
                st[c][e] = s;
                mt = fmaxf(mt, s);
            }
        mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
        const float m_new = fmaxf(m_run, mt);
        const float alpha = exp2f(m_run - m_new);
        float lt = 0.f;
        bf16x8 pf[2][2];
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const float p = exp2f(st[c][e] - m_new);
                lt += p;
                pf[c][e >> 3][e & 7] = (__bf16)p;
            }
        lt += __shfl_xor(lt, 32, 64);
        l_run = l_run * alpha + lt;
        m_run = m_new;
#pragma unroll
        for (int n = 0; n < C::NB; ++n)
#pragma unroll
            for (int e = 0; e < 16; ++e) oacc[n][e] *= alpha;

        // O^T += V^T P^T
#pragma unroll
        for (int n = 0; n < C::NB; ++n) {
            const char* vrow = Vs + (n * 32 + j) * C::V_STRIDE;
#pragma unroll
            for (int c = 0; c < 2; ++c)
#pragma unroll
                for (int s2 = 0; s2 < 2; ++s2) {
                    const int key = c * 32 + 16 * s2 + 4 * g;
                    const u32x2 lo = *reinterpret_cast<const u32x2*>(vrow + key * 2);
                    const u32x2 hi = *reinterpret_cast<const u32x2*>(vrow + (key + 8) * 2);
                    u32x4 w4 = u32x4{lo[0], lo[1], hi[0], hi[1]};
                    const bf16x8 vf = __builtin_bit_cast(bf16x8, w4);
                    oacc[n] = mfma32x32x16(vf, pf[c][s2], oacc[n]);
                }
        }
        if (kt + 1 < nkt) lstore((kt + 1) & 1);
        __syncthreads();
    }

    if (q < S) {
        const float inv = 1.f / l_run;
        bf16_t* orow = O + ((int64_t)b * S + q) * ((int64_t)H * HD) + (int64_t)h * HD;
#pragma unroll
        for (int n = 0; n < C::NB; ++n)
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int hd0 = n * 32 + 8 * t + 4 * g;
                const uint32_t w0 = pack_bf16x2(oacc[n][4 * t] * inv, oacc[n][4 * t + 1] * inv);
                const uint32_t w1 = pack_bf16x2(oacc[n][4 * t + 2] * inv, oacc[n][4 * t + 3] * inv);
                *reinterpret_cast<u32x2*>(orow + hd0) = u32x2{w0, w1};
            }
    }
}

}  // namespace

hipError_t launch_attention(const bf16_t* q, const bf16_t* k, const bf16_t* v, bf16_t* o, int B,
                            int S, int H, int KV, int hd, hipStream_t st) {
    const dim3 grid((S + 127) / 128, H, B);
    const float scale_log2 = 1.4426950408889634f / sqrtf((float)hd);
    if (hd == 128)
        hipLaunchKernelGGL(attn_kernel<128>, grid, dim3(256), 0, st, q, k, v, o, S, H, KV, scale_log2);
    else if (hd == 64)
        hipLaunchKernelGGL(attn_kernel<64>, grid, dim3(256), 0, st, q, k, v, o, S, H, KV, scale_log2);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}
