// Non-causal (bidirectional) grouped-query attention for the refinement pass.
//
// Every query attends to all S keys of its sequence: the refiner revises any
// draft position using context from the whole prompt+draft (paper Sec. 4.2),
// so there is no causal or block mask.  Keys beyond S (tile padding) are the
// only masked entries.
//
// The same kernel serves block-AR drafting (Sec. 3.3): there the queries are
// the Sq rows of one window (the prompt, or one block) and the keys are the
// first n_keys rows of a longer per-layer K/V cache of Skv rows (everything up
// to the window's end).  Every window query sees exactly those keys, which is
// the block-causal mask for a window that is one block or the prompt.  A
// window may also hold the finished block before the current one: its first
// q_split query rows then see only the first n_keys_lo keys (up to their own
// block's end), the others all n_keys.
//
// One workgroup = 4 waves = 128 queries of one (batch, head); each wave owns 32
// queries.  Per tile of KEYS keys, K [KEYS][hd] and V^T [hd][KEYS] are copied
// global -> LDS by buffer loads (NS stages, XOR-swizzled 16-byte chunks).
// Scores are computed transposed, S^T = K Q^T, so that each lane owns one
// query column: the online-softmax statistics stay lane-local (plus one
// exchange with lane^32) and the probabilities feed the next MFMA straight
// from registers as the B operand of O^T = V^T P^T.  V^T arrives from the QKV
// projection with its keys already in the order that operand needs (vt_pos),
// so every fragment is one 16-byte LDS read.
// The running maximum is only moved (and the accumulator rescaled) when a
// tile raises it by more than 2^8 in the exp2 domain; in between,
// probabilities up to 2^8 are accumulated, which the final division by the
// running sum cancels exactly.
#include "common.h"
#include "kernels.h"

namespace {

template <int HD, int KEYS_>
struct AttnCfg {
    static constexpr int KEYS = KEYS_;                  // keys per tile (32 or 64)
    static constexpr int NC = KEYS / 32;                // 32-key chunks per tile
    static constexpr int K_CPR = HD / 8;                // 16-byte chunks per K row
    static constexpr int K_ROW = HD * 2;
    static constexpr int K_BYTES = KEYS * K_ROW;
    static constexpr int V_CPR = KEYS / 8;              // 16-byte chunks per V^T row
    static constexpr int V_ROW = KEYS * 2;
    static constexpr int V_BYTES = HD * V_ROW;
    static constexpr int STAGE = K_BYTES + V_BYTES;
    static constexpr int K_INSTR = K_BYTES / 1024 / 4;  // 1 KB copies per wave per tile
    static constexpr int V_INSTR = V_BYTES / 1024 / 4;
    static constexpr int NB = HD / 32;                  // 32-row blocks of O^T
    static constexpr int NKS = HD / 16;                 // K16 steps over hd
};

// XOR key of the 16-byte chunks of an LDS row of CPR chunks; fragment reads of
// 32 consecutive rows at one logical chunk then hit distinct banks (with
// 4-chunk rows, four consecutive rows share a 256-byte bank line, so the key
// takes the row bits above them).
template <int CPR>
__device__ __forceinline__ int chunk_key(int row) {
    if constexpr (CPR == 16) return row & 15;
    else if constexpr (CPR == 8) return (row & 7) ^ ((row >> 3) & 1);
    else return (row >> 2) & 3;
}

// max / sum of v and its value in lane ^ 32 (v_permlane32_swap: no LDS trip)
__device__ __forceinline__ float xor32_max(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xor32_sum(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int HD, int KEYS, int WPE, int NS>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(WPE))) void attn_kernel(const bf16_t* __restrict__ Q, const bf16_t* K,
                                                   const bf16_t* Vt, bf16_t* __restrict__ O, int Sq, int Skv,
                                                   int n_keys, int q_split, int n_keys_lo, int H, int KV,
                                                   float scale_log2, uint32_t k_bytes, uint32_t v_bytes) {
    using C = AttnCfg<HD, KEYS>;
    static_assert(NS >= 2, "at least two K/V stages");
    __shared__ __attribute__((aligned(16))) char smem[NS * C::STAGE];

    const int tid = threadIdx.x, lane = tid & 63, wave = uniform(tid >> 6);   // scalar: wave-level branches stay branches
    const int g = lane >> 5, j = lane & 31;
    const int qb = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const int kvh = h / (H / KV);
    const int q = qb * 128 + wave * 32 + j;
    const int lim = q < q_split ? n_keys_lo : n_keys;   // keys this lane's query sees
    const int VS = vt_stride(Skv);
    const int wv = wave;

    const bf16_t* Qh = Q + ((int64_t)b * H + h) * Sq * HD;
    // The last K tile reads up to 63 rows past n_keys: later rows of the same
    // head, rows of the next head (all masked), or past the last head into the
    // buffer's one-tile tail.  V^T rows are padded to whole tiles, so V^T
    // reads stay inside their row.
    const buf_rsrc_t k_rsrc = make_rsrc(K, (int)k_bytes);
    const buf_rsrc_t v_rsrc = make_rsrc(Vt, (int)v_bytes);
    const uint32_t k_base = (uint32_t)(((int64_t)b * KV + kvh) * Skv * HD * 2);
    const uint32_t v_base = (uint32_t)(((int64_t)b * KV + kvh) * HD * VS * 2);

    // Per-lane byte offsets of this wave's copies (tile-relative; the key
    // offset of the tile goes into the scalar offset).
    uint32_t k_off[C::K_INSTR], v_off[C::V_INSTR];
    {
        constexpr int KRB = 64 / C::K_CPR;              // K rows per 1 KB block
#pragma unroll
        for (int p = 0; p < C::K_INSTR; ++p) {
            const int row = (wv * C::K_INSTR + p) * KRB + lane / C::K_CPR;
            const int pc = lane % C::K_CPR;
            k_off[p] = k_base + (uint32_t)(row * HD * 2 + ((pc ^ chunk_key<C::K_CPR>(row)) * 16));
        }
        constexpr int VRB = 64 / C::V_CPR;              // V^T rows per 1 KB block
#pragma unroll
        for (int p = 0; p < C::V_INSTR; ++p) {
            const int row = (wv * C::V_INSTR + p) * VRB + lane / C::V_CPR;
            const int pc = lane % C::V_CPR;
            v_off[p] = v_base + (uint32_t)(row * VS * 2 + ((pc ^ chunk_key<C::V_CPR>(row)) * 16));
        }
    }
    const lds_ptr_t lds = (lds_ptr_t)smem;
    typedef __attribute__((address_space(3))) char lds_char;
    typedef __attribute__((address_space(3))) const bf16x8 lds_frag;
    auto issue = [&](int kt, int stage) {
        const int k_soff = kt * C::KEYS * HD * 2, v_soff = kt * C::KEYS * 2;
        const int kd = stage * C::STAGE + wv * C::K_INSTR * 1024;
        const int vd = stage * C::STAGE + C::K_BYTES + wv * C::V_INSTR * 1024;
#pragma unroll
        for (int p = 0; p < C::K_INSTR; ++p)
            lds_dma16_buf(k_rsrc, k_off[p], k_soff, (lds_ptr_t)((lds_char*)lds + kd + p * 1024));
#pragma unroll
        for (int p = 0; p < C::V_INSTR; ++p)
            lds_dma16_buf(v_rsrc, v_off[p], v_soff, (lds_ptr_t)((lds_char*)lds + vd + p * 1024));
    };

    bf16x8 qf[C::NKS];
    {
        const bf16_t* qp = Qh + (int64_t)min(q, Sq - 1) * HD + g * 8;
#pragma unroll
        for (int ks = 0; ks < C::NKS; ++ks) qf[ks] = *reinterpret_cast<const bf16x8*>(qp + ks * 16);
    }

    f32x16 oacc[C::NB];
#pragma unroll
    for (int n = 0; n < C::NB; ++n)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[n][e] = 0.f;
    float m_run = -INFINITY, l_run = 0.f;           // m_run in raw score units

    // Fragment bases: K row c*32 + j, chunk 2ks + g; V^T row n*32 + j,
    // chunk 4c + 2s2 + g.  The XOR key depends on the low row bits only.
    const int kfrag = j * C::K_ROW;
    const int kkey = chunk_key<C::K_CPR>(j);
    const int vfrag = C::K_BYTES + j * C::V_ROW;
    const int vkey = chunk_key<C::V_CPR>(j);

    const int nkt = (n_keys + C::KEYS - 1) / C::KEYS;
    // Tiles kt .. kt + NS - 2 are in flight at the top of tile kt; copies past
    // the last tile repeat it into a stage that is never read, so that every
    // wait below counts the same number of copies.
#pragma unroll
    for (int t = 0; t < NS - 1; ++t) issue(min(t, nkt - 1), t);
    int stage = 0;
    for (int kt = 0; kt < nkt; ++kt) {
        wait_vmcnt<(NS - 2) * (C::K_INSTR + C::V_INSTR)>();   // this wave's copies of tile kt landed
        __syncthreads();                            // everyone's; the stage of tile kt-1 is free
        issue(min(kt + NS - 1, nkt - 1), stage == 0 ? NS - 1 : stage - 1);
        const int sb = stage * C::STAGE;
        stage = stage + 1 == NS ? 0 : stage + 1;
        const int k0 = kt * C::KEYS;

        // S^T for the tile's keys (32-key chunks): lane holds query j, keys
        // c*32 + 8*(e/4) + 4*g + e%4.
        f32x16 st[C::NC];
#pragma unroll
        for (int c = 0; c < C::NC; ++c) {
#pragma unroll
            for (int e = 0; e < 16; ++e) st[c][e] = 0.f;
            // K fragments in batches of four reads issued together, so that the
            // accumulation chain waits for one LDS latency per batch.
#pragma unroll
            for (int k4 = 0; k4 < C::NKS; k4 += 4) {
                bf16x8 kf[4];
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    kf[u] = *(lds_frag*)((lds_char*)lds + sb + c * 32 * C::K_ROW + kfrag + (((2 * (k4 + u) + g) ^ kkey) << 4));
                sched_fence();
#pragma unroll
                for (int u = 0; u < 4; ++u) st[c] = mfma32x32x16(kf[u], qf[k4 + u], st[c]);
            }
        }
        if (k0 + C::KEYS > lim) {                   // keys past the lane's limit are not visible
#pragma unroll
            for (int c = 0; c < C::NC; ++c)
#pragma unroll
                for (int e = 0; e < 16; ++e)
                    if (k0 + c * 32 + 8 * (e >> 2) + 4 * g + (e & 3) >= lim) st[c][e] = -INFINITY;
        }
        float mt = -INFINITY;
#pragma unroll
        for (int c = 0; c < C::NC; ++c)
#pragma unroll
            for (int e = 0; e < 16; ++e) mt = fmaxf(mt, st[c][e]);
        mt = xor32_max(mt);
        if (__any((mt - m_run) * scale_log2 > 8.f)) {
            const float m_new = fmaxf(m_run, mt);
            const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * scale_log2);
            l_run *= alpha;
#pragma unroll
            for (int n = 0; n < C::NB; ++n)
#pragma unroll
                for (int e = 0; e < 16; ++e) oacc[n][e] *= alpha;
            m_run = m_new;
        }
        const float nb = -m_run * scale_log2;
        float lt = 0.f;
        bf16x8 pf[C::NC][2];
#pragma unroll
        for (int c = 0; c < C::NC; ++c)
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2) {
                u32x4 w;
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const float p0 = __builtin_amdgcn_exp2f(fmaf(st[c][8 * s2 + 2 * t], scale_log2, nb));
                    const float p1 = __builtin_amdgcn_exp2f(fmaf(st[c][8 * s2 + 2 * t + 1], scale_log2, nb));
                    lt += p0 + p1;
                    w[t] = pack_bf16x2(p0, p1);
                }
                pf[c][s2] = __builtin_bit_cast(bf16x8, w);
            }
        l_run += lt;

        // O^T += V^T P^T: one 16-byte V^T read per fragment, read in batches
        // of four (two 32-row blocks of O^T)
#pragma unroll
        for (int c = 0; c < C::NC; ++c)
#pragma unroll
            for (int n2 = 0; n2 < C::NB; n2 += 2) {
                bf16x8 vf[2][2];
#pragma unroll
                for (int n = 0; n < 2; ++n)
#pragma unroll
                    for (int s2 = 0; s2 < 2; ++s2)
                        vf[n][s2] = *(lds_frag*)((lds_char*)lds + sb + vfrag + (n2 + n) * 32 * C::V_ROW +
                                                 (((4 * c + 2 * s2 + g) ^ vkey) << 4));
                sched_fence();
#pragma unroll
                for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
                    for (int n = 0; n < 2; ++n) oacc[n2 + n] = mfma32x32x16(vf[n][s2], pf[c][s2], oacc[n2 + n]);
            }
    }

    wait_all_memory();                              // no copy may still land in LDS when the workgroup ends
    l_run = xor32_sum(l_run);
    // O^T accumulators: lane (query j, g) holds features n*32 + 8t + 4g .. +3;
    // after swap_halves16 it holds n*32 + 16g .. +15, stored as two 16-byte
    // writes (every lane takes part in the exchange; only rows q < Sq store).
    const float inv = 1.f / l_run;
    bf16_t* orow = O + ((int64_t)b * Sq + min(q, Sq - 1)) * ((int64_t)H * HD) + (int64_t)h * HD;
#pragma unroll
    for (int n = 0; n < C::NB; ++n) {
        uint32_t p[4][2];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            p[t][0] = pack_bf16x2(oacc[n][4 * t] * inv, oacc[n][4 * t + 1] * inv);
            p[t][1] = pack_bf16x2(oacc[n][4 * t + 2] * inv, oacc[n][4 * t + 3] * inv);
        }
        swap_halves16(p);
        if (q < Sq) {
            bf16_t* dst = orow + n * 32 + 16 * g;
            *reinterpret_cast<u32x4*>(dst) = u32x4{p[0][0], p[0][1], p[2][0], p[2][1]};
            *reinterpret_cast<u32x4*>(dst + 8) = u32x4{p[1][0], p[1][1], p[3][0], p[3][1]};
        }
    }
}

}  // namespace

hipError_t launch_attention(const bf16_t* q, const bf16_t* k, const bf16_t* vt, bf16_t* o, int B,
                            int Sq, int Skv, int n_keys, int H, int KV, int hd, hipStream_t st, int q_split,
                            int n_keys_lo) {
    if (Sq <= 0 || n_keys <= 0 || n_keys > Skv) return hipErrorInvalidValue;
    if (q_split < 0 || q_split > Sq || (q_split > 0 && (n_keys_lo < 1 || n_keys_lo > n_keys)))
        return hipErrorInvalidValue;
    const dim3 grid((Sq + 127) / 128, H, B);
    const float scale_log2 = 1.4426950408889634f / sqrtf((float)hd);
    // byte sizes of the K buffer (with its one-tile tail) and of V^T
    const int64_t kb = ((int64_t)B * KV * Skv + 64) * hd * 2, vb = (int64_t)B * KV * hd * vt_stride(Skv) * 2;
    if (kb >= 0x7fffffff || vb >= 0x7fffffff) return hipErrorInvalidValue;   // 32-bit buffer offsets
    // 32-key tiles in three stages: 161 VGPRs at head_dim 128, so three
    // workgroups (12 waves) share a CU (48 KB of LDS each).
    if (hd == 128)
        hipLaunchKernelGGL((attn_kernel<128, 32, 3, 3>), grid, dim3(256), 0, st, q, k, vt, o, Sq, Skv, n_keys, q_split,
                           n_keys_lo, H, KV, scale_log2, (uint32_t)kb, (uint32_t)vb);
    else if (hd == 64)
        hipLaunchKernelGGL((attn_kernel<64, 32, 3, 3>), grid, dim3(256), 0, st, q, k, vt, o, Sq, Skv, n_keys, q_split,
                           n_keys_lo, H, KV, scale_log2, (uint32_t)kb, (uint32_t)vb);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}
