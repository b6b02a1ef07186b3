// Device-side helpers shared by the refinement-step kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef uint16_t bf16_t;                                              // raw bfloat16 bits
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define DLM_WAVE 64

__device__ __forceinline__ float bf16_to_f32(bf16_t h) {
    return __uint_as_float(((uint32_t)h) << 16);
}

// float -> bf16, round to nearest even (v_cvt_pk_bf16_f32 on gfx950; NaN
// stays NaN).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __builtin_bit_cast(bf16_t, (__bf16)f);
#else
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u) return (bf16_t)((u >> 16) | ((u & 0xffffu) ? 0x40u : 0u));
    u += 0x7fffu + ((u >> 16) & 1u);
    return (bf16_t)(u >> 16);
#endif
}

// Two floats -> packed bf16 pair (lo in bits 0-15), one conversion instruction.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
#if defined(__HIP_DEVICE_COMPILE__)
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    const f32x2_t v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
#else
    return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
#endif
}

// gfx950 intrinsics used by the kernels.  Their bodies exist only in the
// device compilation pass; the host pass sees empty functions.
typedef __attribute__((address_space(3))) void* lds_ptr_t;

// 16 bytes per lane from global memory straight into LDS: lane L of the wave
// writes bytes [16L, 16L+16) of the block starting at `lds` (wave-uniform).
__device__ __forceinline__ void lds_dma16(const void* src, void* lds) {
#if defined(__HIP_DEVICE_COMPILE__)
    __builtin_amdgcn_global_load_lds(src, (lds_ptr_t)lds, 16, 0, 0);
#endif
}
// Raw buffer resource over a byte range starting at `base` (wave-uniform):
// loads address base + voffset + soffset, with 32-bit offsets.
#if defined(__HIP_DEVICE_COMPILE__)
typedef __amdgpu_buffer_rsrc_t buf_rsrc_t;
#else
struct buf_rsrc_t {
    uint32_t w[4];
};
#endif
__device__ __forceinline__ buf_rsrc_t make_rsrc(const void* base, int bytes = 0x7fffffff) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, 0x00020000);
#else
    return buf_rsrc_t{};
#endif
}
// Buffer form of lds_dma16: lane L reads 16 bytes at voffset(L) + soffset and
// writes them to bytes [16L, 16L+16) of the LDS block at `lds`.
__device__ __forceinline__ void lds_dma16_buf(buf_rsrc_t r, uint32_t voffset, int soffset, lds_ptr_t lds) {
#if defined(__HIP_DEVICE_COMPILE__)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, lds, 16, (int)voffset, soffset, 0, 0);
#endif
}
// Wait until at most N LDS operations of this wave are outstanding.
template <int N>
__device__ __forceinline__ void wait_lgkmcnt() {
    static_assert(N >= 0 && N < 16, "lgkmcnt range");
#if defined(__HIP_DEVICE_COMPILE__)
    __builtin_amdgcn_s_waitcnt(0xC07F | (N << 8));
#endif
}
// Wait until every outstanding memory operation of this wave has completed.
__device__ __forceinline__ void wait_all_memory() {
#if defined(__HIP_DEVICE_COMPILE__)
    __builtin_amdgcn_s_waitcnt(0);
#endif
}
// Wait until at most N vector-memory operations of this wave are outstanding
// (gfx9 s_waitcnt encoding: vmcnt in bits 3:0 and 15:14; other counters left at max).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
#if defined(__HIP_DEVICE_COMPILE__)
    __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
#endif
}
__device__ __forceinline__ int uniform(int v) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __builtin_amdgcn_readfirstlane(v);
#else
    return v;
#endif
}
// Scheduling hint: `n` instructions of class `mask` next (0x8 MFMA, 0x100 LDS read).
template <int MASK, int N>
__device__ __forceinline__ void sched_group() {
#if defined(__HIP_DEVICE_COMPILE__)
    __builtin_amdgcn_sched_group_barrier(MASK, N, 0);
#endif
}

// Scheduling fence: the compiler moves no instruction across it.
// Load of an int that no thread writes during the kernel, through the
// constant address space: with a wave-uniform address it becomes a scalar
// load (counted by lgkmcnt, not behind the vector-memory queue).
__device__ __forceinline__ int ld_const(const int* p) {
#if defined(__HIP_DEVICE_COMPILE__)
    return *(const __attribute__((address_space(4))) int*)p;
#else
    return *p;
#endif
}

__device__ __forceinline__ void sched_fence() {
#if defined(__HIP_DEVICE_COMPILE__)
    __builtin_amdgcn_sched_barrier(0);
#endif
}

// Workgroup barrier without the memory-model fence of __syncthreads (whose
// release half also waits for every copy into LDS still in flight): it only
// makes this wave's LDS reads complete first.  Copies that other waves will
// read must be awaited by count before it; the empty asm statements keep the
// compiler from moving memory accesses across it.
__device__ __forceinline__ void lds_barrier() {
#if defined(__HIP_DEVICE_COMPILE__)
    __builtin_amdgcn_s_waitcnt(0xC07F);      // lgkmcnt(0)
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
#endif
}

// Row segment of a transposed 32x32 accumulator block, for wide stores.  In
// the transposed layout lane (r, h) = (lane % 32, lane / 32) holds columns
// 8q + 4h .. 8q + 4h + 3 (q = 0..3) of row r; p[q] holds them as two packed
// bf16 pairs.  Exchanging q = 2, 3 of lanes 0-31 with q = 0, 1 of lanes 32-63
// (v_permlane32_swap) leaves lane (r, h) with columns 16h .. 16h + 15 of row
// r in the order p[0], p[2], p[1], p[3]: two 16-byte stores per lane, a
// 32-byte run of each row per pair of store instructions.
__device__ __forceinline__ void swap_halves16(uint32_t (&p)[4][2]) {
#if defined(__HIP_DEVICE_COMPILE__)
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const auto a = __builtin_amdgcn_permlane32_swap(p[0][k], p[2][k], false, false);
        const auto b = __builtin_amdgcn_permlane32_swap(p[1][k], p[3][k], false, false);
        p[0][k] = a[0];
        p[2][k] = a[1];
        p[1][k] = b[0];
        p[3][k] = b[1];
    }
#endif
}

__device__ __forceinline__ f32x16 mfma32x32x16(const bf16x8& a, const bf16x8& b, const f32x16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Wave-wide reductions (64 lanes).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}

// 1 / sqrt(mean(x^2) + eps) of a row held by a workgroup of up to 4 waves,
// from each thread's partial sum of squares: per-wave sums, then the waves in
// order (a fixed order: every kernel that normalises a row this way gets the
// same bits for the same row).
__device__ __forceinline__ float block_rms_scale(float ss, int d, float eps) {
    __shared__ float red[4];
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    float tot = 0.f;
    const int nw = blockDim.x >> 6;
    for (int w = 0; w < nw; ++w) tot += red[w];
    return 1.f / sqrtf(tot / (float)d + eps);
}

// hr = bf16(xr * r * g) for the chunks of 8 this thread owns in a row
// normalised by a workgroup (chunk i*8 .. i*8+7 for i = thread + k * threads).
__device__ __forceinline__ void rms_store_row(const float* xr, const bf16_t* __restrict__ g, bf16_t* __restrict__ hr,
                                              int d, float r) {
    for (int i = threadIdx.x * 8; i < d; i += blockDim.x * 8) {
        const f32x4 a = *reinterpret_cast<const f32x4*>(xr + i);
        const f32x4 b = *reinterpret_cast<const f32x4*>(xr + i + 4);
        const u32x4 gg = *reinterpret_cast<const u32x4*>(g + i);
        float gv[8];
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            gv[2 * w] = __uint_as_float(gg[w] << 16);
            gv[2 * w + 1] = __uint_as_float(gg[w] & 0xffff0000u);
        }
        u32x4 o;
        o[0] = pack_bf16x2(a[0] * r * gv[0], a[1] * r * gv[1]);
        o[1] = pack_bf16x2(a[2] * r * gv[2], a[3] * r * gv[3]);
        o[2] = pack_bf16x2(b[0] * r * gv[4], b[1] * r * gv[5]);
        o[3] = pack_bf16x2(b[2] * r * gv[6], b[3] * r * gv[7]);
        *reinterpret_cast<u32x4*>(hr + i) = o;
    }
}

// Wave-wide reductions on DPP lane moves (no LDS traffic), the total read
// from lane 63: within each quad, then 8 and 16 lanes (mirrors), then rows
// 0+1 into row 1 and rows 2+3 into row 3 (broadcast of lane 15 of the row
// below), then row 3 += lane 31.  A fixed order, so the result is the same on
// every call with the same inputs.
template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ float dpp_f(float v) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, ROWS, 0xF, false));
#else
    return v;
#endif
}
__device__ __forceinline__ float wave_sum_dpp(float v) {
#if defined(__HIP_DEVICE_COMPILE__)
    v += dpp_f<0xB1>(v);            // quad_perm [1,0,3,2]
    v += dpp_f<0x4E>(v);            // quad_perm [2,3,0,1]
    v += dpp_f<0x141>(v);           // row_half_mirror
    v += dpp_f<0x140>(v);           // row_mirror
    v += dpp_f<0x142, 0xA>(v);      // row_bcast:15 into rows 1, 3
    v += dpp_f<0x143, 0xC>(v);      // row_bcast:31 into rows 2, 3
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
#else
    return v;
#endif
}
__device__ __forceinline__ float wave_max_dpp(float v) {
#if defined(__HIP_DEVICE_COMPILE__)
    v = fmaxf(v, dpp_f<0xB1>(v));
    v = fmaxf(v, dpp_f<0x4E>(v));
    v = fmaxf(v, dpp_f<0x141>(v));
    v = fmaxf(v, dpp_f<0x140>(v));
    // rows outside the mask keep v (max with -inf from the zero-filled move
    // would be wrong for all-negative inputs), hence the explicit select
    const float b15 = __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, v), __builtin_bit_cast(int, v), 0x142, 0xA, 0xF, false));
    v = fmaxf(v, b15);
    const float b31 = __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, v), __builtin_bit_cast(int, v), 0x143, 0xC, 0xF, false));
    v = fmaxf(v, b31);
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
#else
    return v;
#endif
}

// Online-softmax partial over a set of logits: running max m, the lowest index
// attaining it, and s = sum exp(z - m).  merge() is associative up to float
// rounding and keeps the lower index on equal maxima.
struct SoftmaxPartial {
    float m;
    int32_t idx;
    float s;
};

__device__ __forceinline__ SoftmaxPartial sp_merge(SoftmaxPartial a, SoftmaxPartial b) {
    SoftmaxPartial r;
    if (b.m > a.m || (b.m == a.m && b.idx < a.idx)) {
        r.m = b.m;
        r.idx = b.idx;
    } else {
        r.m = a.m;
        r.idx = a.idx;
    }
    float sa = (a.s == 0.f) ? 0.f : a.s * __expf(a.m - r.m);
    float sb = (b.s == 0.f) ? 0.f : b.s * __expf(b.m - r.m);
    r.s = sa + sb;
    return r;
}
