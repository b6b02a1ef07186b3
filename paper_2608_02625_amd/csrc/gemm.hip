// bf16 MFMA GEMM for gfx950 with fused epilogues.
//
// C[M x N] = A[M x K] * B[N x K]^T, fp32 accumulation, both operands K-contiguous.
// A workgroup owns a BM x BN tile: 4 waves in a 2x2 grid or 8 waves in a 2x4
// grid (two per SIMD), each wave a grid of 32x32 accumulators fed by
// v_mfma_f32_32x32x16_bf16.  K advances BK at a time through LDS stages filled
// straight from global memory by buffer loads (no register staging) while the
// MFMAs of earlier K tiles run.  Two schedules: every wave interleaves its
// fragment reads with its MFMAs, or (ping-pong, 8 waves) the two waves of a
// SIMD take turns, one multiplying a whole K tile while the other copies and
// reads the next.
// LDS rows are BK*2 bytes with 16-byte chunks XOR-swizzled by row bits so that
// fragment reads of 32 consecutive rows spread over all banks.
//
// Grouped mode runs one GEMM per expert over a device-built tile table; the A
// rows of a group may be gathered through an index array (token -> expert
// rows), so the routed activations are never copied.
//
// Workgroup ids are remapped so that each of the 8 XCDs (which receive
// workgroups round-robin) processes a contiguous range of tiles; within that
// range dense GEMMs raster group_m row-tiles at a time to keep operands in L2.
#include <algorithm>
#include <atomic>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kMaxDevices = 64;

template <int BM, int BN, int BK, int SA, int SB, int NW>
struct TileCfg {
    static constexpr int NT = NW * 64;                   // threads
    static constexpr int WM = BM / 2, WN = BN / (NW / 2);
    static constexpr int TM = WM / 32, TN = WN / 32;
    static constexpr int ROW = BK * 2;                   // bytes per LDS tile row
    static constexpr int CPR = BK / 8;                   // 16-byte chunks per row
    static constexpr int KS = BK / 16;                   // MFMA K steps per tile
    static constexpr int A_BYTES = BM * ROW, B_BYTES = BN * ROW;
    static constexpr int LDS = SA * A_BYTES + SB * B_BYTES;
    static constexpr int A_INSTR = A_BYTES / 1024 / NW;  // 1 KB DMA blocks per wave
    static constexpr int B_INSTR = B_BYTES / 1024 / NW;
    // The operand with fewer stages is copied first in every round of copies
    // (S = shallow, D = deep).  Waiting until at most N copies are pending
    // (copies complete in order) then guarantees:
    //   N_TOP:  K tile 0 of both operands landed (after the first round);
    //   N_LOOP: K tile kt+1 of both landed, at the barrier of tile kt.
    static constexpr int SS = SA < SB ? SA : SB, SD = SA < SB ? SB : SA;
    static constexpr int NI_S = SA <= SB ? A_INSTR : B_INSTR, NI_D = SA <= SB ? B_INSTR : A_INSTR;
    static constexpr int N_TOP = (SS - 1) * NI_S + (SD - 1) * NI_D;
    static constexpr int CNT_S = NI_D + (SS - 2) * (NI_S + NI_D), CNT_D = (SD - 2) * (NI_S + NI_D);
    static constexpr int N_LOOP = CNT_S < CNT_D ? CNT_S : CNT_D;
    static_assert(SS >= 2, "at least two stages per operand");
};

// XOR key of the 16-byte chunks of a tile row: consecutive rows read by one
// MFMA fragment land in distinct LDS banks (checked: no bank conflicts).
template <int CPR>
__device__ __forceinline__ int swz_key(int row) {
    if constexpr (CPR == 8) return (row & 7) ^ ((row >> 3) & 1);
    else return ((row >> 1) & 3) ^ ((row >> 3) & 1);
}

// Byte offset of logical 16-byte chunk `chunk` of tile row `row`.
template <int CPR>
__device__ __forceinline__ int swz(int row, int chunk) {
    return row * (CPR * 16) + ((chunk ^ swz_key<CPR>(row)) << 4);
}

// QKV projection, computed transposed: rows = q/k/v features, columns =
// tokens.  A lane then holds, per accumulator, 4 consecutive features of one
// token (8-byte stores into Q [B][H][S][hd] and K [B][KV][S][hd]; V goes to the
// transposed layout V^T of kernels.h, consecutive lanes = consecutive keys), and a
// wave's 128 rows cover whole heads, so the RoPE partners (i, i + hd/2) are in
// the same lane, accumulator rows i and i + hd/64 (rotate-half, applied in
// fp32 before rounding).
template <int TM, int TN, int HD>
__device__ __forceinline__ void qkv_epilogue(const GemmArgs& a, const f32x16 (&acc)[TM][TN], int m0, int n0,
                                             int lrow0, int lcol0) {
    constexpr int HALF = HD / 2, SPH = HD / 32, POFF = HD / 64;
    const int Hq = a.n_heads * HD, Hk = a.n_kv * HD;
    const int S = a.seq, SK = a.kv_seq;
    // A wave's 128 rows start on a head boundary, and the Q/K/V boundaries are
    // head boundaries: the wave is wholly inside Q, K or V (or past M).
    const int wrow = m0 + (lrow0 & ~127);
    if (wrow >= a.M) return;
    const bool rotate = wrow < Hq + Hk;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        const int t_raw = n0 + lcol0 + j * 32;                // token
        const bool live = t_raw < a.N;
        const int t = live ? t_raw : a.N - 1;                 // lanes past the end compute, then store nothing
        const int b = t / S, s = t - b * S;
        const int sk = s + a.pos0;                            // position in K / V^T and the RoPE table
        if (rotate) {
            // (cos, sin) of the lane's 4 consecutive pairs for each first-half
            // 32-row block and each group q, all loaded before use.
            float4 cs[POFF][4][2];
#pragma unroll
            for (int ih = 0; ih < POFF; ++ih)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int r0 = (lrow0 & 127) + ih * 32 + 8 * q;       // row within the head pair block
                    const float4* p = reinterpret_cast<const float4*>(a.rope + sk * HALF + (r0 % HALF));
                    cs[ih][q][0] = p[0];
                    cs[ih][q][1] = p[1];
                }
            // Per 32-feature block: the rotated features of this lane's token,
            // packed, then exchanged between lane halves (swap_halves16) so
            // that each lane writes 16 consecutive features as two 16-byte
            // stores.
            const int half = (lrow0 >> 2) & 1;                  // lane / 32
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                uint32_t p[4][2];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int ih = (i % SPH) % POFF;
                    const float4 c01 = cs[ih][q][0], c23 = cs[ih][q][1];
                    const float cz[4] = {c01.x, c01.z, c23.x, c23.z};
                    const float sn[4] = {c01.y, c01.w, c23.y, c23.w};
                    float v[4];
                    if ((i % SPH) < POFF) {
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            v[r] = acc[i][j][4 * q + r] * cz[r] - acc[(i + POFF) % TM][j][4 * q + r] * sn[r];
                    } else {
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            v[r] = acc[i][j][4 * q + r] * cz[r] + acc[(i + TM - POFF) % TM][j][4 * q + r] * sn[r];
                    }
                    p[q][0] = pack_bf16x2(v[0], v[1]);
                    p[q][1] = pack_bf16x2(v[2], v[3]);
                }
                swap_halves16(p);
                if (live) {
                    const int fb = m0 + (lrow0 & ~4) + i * 32 + 16 * half;   // first of this lane's 16 features
                    const int hi0 = fb % HD;
                    bf16_t* dst = fb < Hq ? a.q + (((int64_t)b * a.n_heads + fb / HD) * S + s) * HD + hi0
                                          : a.k + (((int64_t)b * a.n_kv + (fb - Hq) / HD) * SK + sk) * HD + hi0;
                    *reinterpret_cast<u32x4*>(dst) = u32x4{p[0][0], p[0][1], p[2][0], p[2][1]};
                    *reinterpret_cast<u32x4*>(dst + 8) = u32x4{p[1][0], p[1][1], p[3][0], p[3][1]};
                }
            }
        } else if (live) {
            // V^T: per accumulator 4 rows (features) of one key column
            const int vs = vt_stride(SK);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int fv = m0 + lrow0 + i * 32 + 8 * q - Hq - Hk;
                    bf16_t* col = a.v + ((int64_t)(b * a.n_kv + fv / HD) * HD + fv % HD) * vs + vt_pos(sk);
#pragma unroll
                    for (int r = 0; r < 4; ++r) col[(int64_t)r * vs] = f32_to_bf16(acc[i][j][4 * q + r]);
                }
        }
    }
}

template <int BM, int BN, int BK, int SA, int SB, int NW, int EPI, bool GROUPED, bool PP>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(NW / 4))) void gemm_kernel(GemmArgs a) {
    using T = TileCfg<BM, BN, BK, SA, SB, NW>;
    __shared__ __attribute__((aligned(16))) char smem[T::LDS];

    const int tid = threadIdx.x, lane = tid & 63, wave = uniform(tid >> 6);   // scalar: wave-level branches stay branches
    const int wm = wave / (NW / 2), wn = wave % (NW / 2);
    const int tiles_n = (a.N + BN - 1) / BN;

    // ---------------------------------------------------------------- tiles
    // Persistent: workgroup w runs on XCD w % 8 (workgroups are dealt to the
    // XCDs round-robin; the grid is a multiple of 8) and walks that XCD's
    // contiguous share of the tiles with a stride of grid/8, so operands shared
    // by neighbouring tiles stay in that XCD's L2.
    const int tiles_m_or_listed = GROUPED ? *a.n_tiles : (a.M + BM - 1) / BM;
    const int total = tiles_m_or_listed * tiles_n;
    const int chunk = (total + 7) >> 3;
    const int x_end = min(((int)blockIdx.x & 7) * chunk + chunk, total);
    const int stride = (int)gridDim.x >> 3;
    int L = ((int)blockIdx.x & 7) * chunk + ((int)blockIdx.x >> 3);
    if (L >= x_end) return;
    struct TileIdx {
        int g, m0, row_base, rows, n0;
    };
    auto decode = [&](int L) {
        int ti, tn;
        if (GROUPED || a.group_m <= 1) {
            ti = L / tiles_n;
            tn = L - ti * tiles_n;
        } else {
            const int tiles_m = tiles_m_or_listed;
            const int per_group = a.group_m * tiles_n;
            const int grp = L / per_group;
            const int first_m = grp * a.group_m;
            const int gsz = min(tiles_m - first_m, a.group_m);
            const int r = L - grp * per_group;
            ti = first_m + r % gsz;
            tn = r / gsz;
        }
        TileIdx t;
        if (GROUPED) {
            // The tile table and group offsets are read-only for the whole
            // launch: scalar loads, no wait behind copies in flight.
            const int* tab = reinterpret_cast<const int*>(a.tile_tab) + 2 * ti;
            t.g = uniform(ld_const(tab));
            t.m0 = uniform(ld_const(tab + 1));
            t.row_base = uniform(ld_const(a.grp_off + t.g));
            t.rows = uniform(ld_const(a.grp_off + t.g + 1)) - t.row_base;
        } else {
            t.g = 0;
            t.m0 = ti * BM;
            t.row_base = 0;
            t.rows = a.M;
        }
        t.n0 = tn * BN;
        return t;
    };

    // ---------------------------------------------------------------- main loop
    // Operands go global -> LDS directly (buffer_load_dwordx4 ... lds): one
    // instruction per wave fills a contiguous 1 KB block of tile rows, lane L
    // writing bytes [16L, 16L+16).  A lane's 32-bit byte offset into its
    // operand is fixed for the whole K loop and K advances through the scalar
    // offset, so the copies cost no vector ALU work.  The XOR swizzle of the
    // 16-byte chunks is applied on the global side: the lane that fills
    // physical chunk pc of row r fetches logical chunk pc ^ key(r).
    // LDS = [A stage 0 .. SA-1 | B stage 0 .. SB-1]; fragment reads are a
    // per-lane base plus a compile-time offset.
    constexpr int CPR = T::CPR;
    constexpr int RPB = 64 / CPR;                               // tile rows per 1 KB block
    constexpr int B_BASE = SA * T::A_BYTES;
    const int wv = wave;
    const int rin = lane / CPR, pc = lane % CPR;
    const bool gather = GROUPED && a.a_rows != nullptr;
    buf_rsrc_t a_rsrc, b_rsrc;
    uint32_t a_off[T::A_INSTR], b_off[T::B_INSTR];
    auto setup_a = [&](const TileIdx& t) {
        a_rsrc = make_rsrc(gather ? a.A : a.A + (int64_t)(t.row_base + t.m0) * a.lda);
#pragma unroll
        for (int p = 0; p < T::A_INSTR; ++p) {
            const int tr = (wv * T::A_INSTR + p) * RPB + rin;     // row within the tile
            const int r = min(t.m0 + tr, t.rows - 1);
            const int64_t grow = gather ? (int64_t)a.a_rows[t.row_base + r] : (int64_t)(r - t.m0);
            a_off[p] = (uint32_t)(grow * a.lda * 2) + (uint32_t)((pc ^ swz_key<CPR>(tr)) * 16);
        }
    };
    auto setup_b = [&](const TileIdx& t) {
        const bf16_t* Bg = a.B + (GROUPED ? (int64_t)t.g * a.b_group_stride : 0);
        b_rsrc = make_rsrc(Bg + (int64_t)t.n0 * a.ldb);
#pragma unroll
        for (int p = 0; p < T::B_INSTR; ++p) {
            const int tr = (wv * T::B_INSTR + p) * RPB + rin;
            const int n = min(t.n0 + tr, a.N - 1) - t.n0;
            b_off[p] = (uint32_t)((int64_t)n * a.ldb * 2) + (uint32_t)((pc ^ swz_key<CPR>(tr)) * 16);
        }
    };
    const lds_ptr_t lds = (lds_ptr_t)smem;
    typedef __attribute__((address_space(3))) char lds_char;
    typedef __attribute__((address_space(3))) const bf16x8 lds_frag;
    auto lds_at = [&](int off) { return (lds_ptr_t)((lds_char*)lds + off); };
    auto issue_a = [&](int kt, int stage) {                      // A of K tile kt -> A stage
        const int dst = stage * T::A_BYTES + wv * T::A_INSTR * 1024;
#pragma unroll
        for (int p = 0; p < T::A_INSTR; ++p) lds_dma16_buf(a_rsrc, a_off[p], kt * (BK * 2), lds_at(dst + p * 1024));
    };
    auto issue_b = [&](int kt, int stage) {
        const int dst = B_BASE + stage * T::B_BYTES + wv * T::B_INSTR * 1024;
#pragma unroll
        for (int p = 0; p < T::B_INSTR; ++p) lds_dma16_buf(b_rsrc, b_off[p], kt * (BK * 2), lds_at(dst + p * 1024));
    };
    // One round of copies: the shallow operand first (see TileCfg).
    auto issue = [&](int kt_a, int st_a, int kt_b, int st_b) {
        if constexpr (SA <= SB) {
            issue_a(kt_a, st_a);
            issue_b(kt_b, st_b);
        } else {
            issue_b(kt_b, st_b);
            issue_a(kt_a, st_a);
        }
    };
    auto prologue = [&](int nk) {                                // first K tiles of a tile, stages 0..
#pragma unroll
        for (int t = 0; t < T::SD; ++t) {
            if constexpr (SA <= SB) {
                if (t < SA) issue_a(min(t, nk - 1), t);
                issue_b(min(t, nk - 1), t);
            } else {
                if (t < SB) issue_b(min(t, nk - 1), t);
                issue_a(min(t, nk - 1), t);
            }
        }
    };

    f32x16 acc[T::TM][T::TN];

    // Fragment step ks of a tile: lanes 0-31 take K chunk 2ks, lanes 32-63
    // chunk 2ks+1, of rows base + (lane & 31).  The swizzle key depends on the
    // low 4 row bits only, so rows +32i share the lane's base offset.
    // Chunk 2ks + h of a row sits at byte ((2ks + h) ^ key) * 16 of the row,
    // i.e. at (slot-0 offset) ^ (ks * 32): one XOR per slot and operand.
    const int fa0 = swz<CPR>(wm * T::WM + (lane & 31), lane >> 5);
    const int fb0 = swz<CPR>(wn * T::WN + (lane & 31), lane >> 5);
    bf16x8 ra[T::KS][T::TM], rb[T::KS][T::TN];
    // Per-lane bases of the stages being read: fa_s = fa0 + stage * A_BYTES
    // (the stage term sits above bit 14, so the slot XOR below commutes with it).
    int fa_s = fa0, fb_s = B_BASE + fb0;
    auto set_stage = [&](int st_a, int st_b) {
        fa_s = fa0 + st_a * T::A_BYTES;
        fb_s = B_BASE + fb0 + st_b * T::B_BYTES;
    };
    auto read_slot = [&](int ks) {                               // fragments of step ks
        const int fa = fa_s ^ (ks * 32), fb = fb_s ^ (ks * 32);
#pragma unroll
        for (int i = 0; i < T::TM; ++i)
            ra[ks][i] = *(lds_frag*)((lds_char*)lds + fa + i * 32 * T::ROW);
#pragma unroll
        for (int j = 0; j < T::TN; ++j)
            rb[ks][j] = *(lds_frag*)((lds_char*)lds + fb + j * 32 * T::ROW);
    };
    // The SwiGLU epilogue, and the bf16 one under the ping-pong schedule, take
    // the accumulators transposed (operands swapped): a lane then holds 4
    // consecutive output columns of one row, stored as one 8-byte write (a
    // quarter of the store instructions; under ping-pong the epilogue runs
    // inside a memory phase, where that count matters).  The other epilogues
    // keep rows in the accumulator's 4-element groups (consecutive lanes =
    // consecutive columns: fully coalesced 2-row accesses; measured faster for
    // the residual read-modify-write).
    constexpr bool TACC = EPI == EPI_SWIGLU || (PP && EPI == EPI_BF16);
    auto mfmas = [&](int ks) {
#pragma unroll
        for (int i = 0; i < T::TM; ++i)
#pragma unroll
            for (int j = 0; j < T::TN; ++j)
                acc[i][j] = TACC ? mfma32x32x16(rb[ks][j], ra[ks][i], acc[i][j])
                                 : mfma32x32x16(ra[ks][i], rb[ks][j], acc[i][j]);
    };
    constexpr int NR = T::TM + T::TN, NM = T::TM * T::TN;
    constexpr int PRE = T::KS / 2;          // fragment steps of a tile run before its barrier

    // ---------------------------------------------------------------- epilogues
    auto epilogue = [&](const int m0, const int rows, const int row_base, const int n0) __attribute__((always_inline)) {
        // TACC: acc[i][j][4q + r] holds C[row][col] with
        //   row = wm*WM + i*32 + lane%32,  col = wn*WN + j*32 + 8q + 4*(lane/32) + r.
        // otherwise acc[i][j][e] holds C[row][col] with
        //   row = wm*WM + i*32 + 8*(e/4) + 4*(lane/32) + e%4,  col = wn*WN + j*32 + lane%32.
        // Lane terms from an opaque copy of the lane id: computed here, not
        // hoisted out of the tile loop into registers live across the K loop.
        int lane = threadIdx.x & 63;
        asm volatile("" : "+v"(lane));
        const int lrow0 = wm * T::WM + 4 * (lane >> 5);
        const int lcol0 = wn * T::WN + (lane & 31);
        const int trow = m0 + wm * T::WM + (lane & 31);              // TACC row of block i = 0
        const int tcol = n0 + wn * T::WN + 4 * (lane >> 5);          // TACC column of j = 0, q = 0
        // 4-column groups are stored whole when they lie inside N and rows are
        // 16-byte (f32) / 8-byte (bf16) aligned.
        const bool vec = (a.ldo & 3) == 0;
        const bool full_tile = m0 + BM <= rows && n0 + BN <= a.N;

        if constexpr (EPI == EPI_BF16 && TACC) {
            // Rows of 32-column blocks: after swap_halves16 a lane holds 16
            // consecutive columns of its row, stored as two 16-byte writes
            // (whole 32-byte runs: fewer partially written cache lines than
            // 8-byte stores, which the store path pays for per line).  The
            // exchange is done by every lane of the wave; rows past the end
            // only skip their stores.
            const bool wide = (a.ldo & 7) == 0;
            const int half = lane >> 5;
#pragma unroll
            for (int i = 0; i < T::TM; ++i) {
                const int r = trow + i * 32;
                bf16_t* orow = reinterpret_cast<bf16_t*>(a.out) + (GROUPED ? (int64_t)row_base + r : r) * a.ldo;
#pragma unroll
                for (int j = 0; j < T::TN; ++j) {
                    const int cb = n0 + wn * T::WN + j * 32;           // first column of the block
                    if (wide && cb + 32 <= a.N) {
                        uint32_t p[4][2];
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            p[q][0] = pack_bf16x2(acc[i][j][4 * q], acc[i][j][4 * q + 1]);
                            p[q][1] = pack_bf16x2(acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
                        }
                        swap_halves16(p);
                        if (r < rows) {
                            bf16_t* dst = orow + cb + 16 * half;
                            *reinterpret_cast<u32x4*>(dst) = u32x4{p[0][0], p[0][1], p[2][0], p[2][1]};
                            *reinterpret_cast<u32x4*>(dst + 8) = u32x4{p[1][0], p[1][1], p[3][0], p[3][1]};
                        }
                    } else if (r < rows) {
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const int c = tcol + j * 32 + 8 * q;
                            const float v[4] = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                                                acc[i][j][4 * q + 3]};
                            if (vec && c + 3 < a.N) {
                                *reinterpret_cast<u32x2*>(orow + c) = u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
                            } else {
#pragma unroll
                                for (int t = 0; t < 4; ++t)
                                    if (c + t < a.N) orow[c + t] = f32_to_bf16(v[t]);
                            }
                        }
                    }
                }
            }
        } else if constexpr (EPI == EPI_RESID) {
            // out[row][col] += acc: per 32-row block all 16 x TN loads are issued
            // before the adds and stores.
            float* out = reinterpret_cast<float*>(a.out);
#pragma unroll
            for (int i = 0; i < T::TM; ++i) {
                float old[16][T::TN];
                const int rb = m0 + lrow0 + i * 32;
                if (full_tile) {
#pragma unroll
                    for (int e = 0; e < 16; ++e)
#pragma unroll
                        for (int j = 0; j < T::TN; ++j)
                            old[e][j] = out[(int64_t)(rb + 8 * (e >> 2) + (e & 3)) * a.ldo + n0 + lcol0 + j * 32];
#pragma unroll
                    for (int e = 0; e < 16; ++e)
#pragma unroll
                        for (int j = 0; j < T::TN; ++j)
                            out[(int64_t)(rb + 8 * (e >> 2) + (e & 3)) * a.ldo + n0 + lcol0 + j * 32] =
                                old[e][j] + acc[i][j][e];
                } else {
#pragma unroll
                    for (int e = 0; e < 16; ++e)
#pragma unroll
                        for (int j = 0; j < T::TN; ++j) {
                            const int r = rb + 8 * (e >> 2) + (e & 3), c = n0 + lcol0 + j * 32;
                            old[e][j] = (r < rows && c < a.N) ? out[(int64_t)r * a.ldo + c] : 0.f;
                        }
#pragma unroll
                    for (int e = 0; e < 16; ++e)
#pragma unroll
                        for (int j = 0; j < T::TN; ++j) {
                            const int r = rb + 8 * (e >> 2) + (e & 3), c = n0 + lcol0 + j * 32;
                            if (r < rows && c < a.N) out[(int64_t)r * a.ldo + c] = old[e][j] + acc[i][j][e];
                        }
                }
            }
        } else if constexpr (EPI == EPI_BF16 || EPI == EPI_F32 || EPI == EPI_F32_T) {
#pragma unroll
            for (int i = 0; i < T::TM; ++i)
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int rl = m0 + lrow0 + i * 32 + 8 * (e >> 2) + (e & 3);
                    if (rl >= rows) continue;
                    const int64_t orow = GROUPED ? (int64_t)row_base + rl : rl;
#pragma unroll
                    for (int j = 0; j < T::TN; ++j) {
                        const int c = n0 + lcol0 + j * 32;
                        if (c >= a.N) continue;
                        const float v = acc[i][j][e];
                        if constexpr (EPI == EPI_BF16)
                            reinterpret_cast<bf16_t*>(a.out)[orow * a.ldo + c] = f32_to_bf16(v);
                        else if constexpr (EPI == EPI_F32)
                            reinterpret_cast<float*>(a.out)[orow * a.ldo + c] = v;
                        else
                            reinterpret_cast<float*>(a.out)[(int64_t)c * a.ldo + orow] = v;
                    }
                }
        } else if constexpr (EPI == EPI_SWIGLU) {
            // Physical columns alternate 32 gate / 32 up: blocks (j, j+1) hold the
            // gate and up values of the same 32 features.  As for the bf16 rows,
            // swap_halves16 gives each lane 16 consecutive features, stored as
            // two 16-byte writes.
            const bool wide = (a.ldo & 7) == 0;
            const int half = lane >> 5;
#pragma unroll
            for (int i = 0; i < T::TM; ++i) {
                const int r = trow + i * 32;
                bf16_t* orow = reinterpret_cast<bf16_t*>(a.out) + (GROUPED ? (int64_t)row_base + r : r) * a.ldo;
#pragma unroll
                for (int j = 0; j < T::TN; j += 2) {
                    const int c0 = n0 + wn * T::WN + j * 32;                // first gate column of the pair
                    if (c0 >= a.N) continue;
                    uint32_t p[4][2];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        float hv[4];
#pragma unroll
                        for (int t = 0; t < 4; ++t) {
                            const float gt = acc[i][j][4 * q + t], up = acc[i][j + 1][4 * q + t];
                            hv[t] = gt * __builtin_amdgcn_rcpf(1.f + __expf(-gt)) * up;
                        }
                        p[q][0] = pack_bf16x2(hv[0], hv[1]);
                        p[q][1] = pack_bf16x2(hv[2], hv[3]);
                    }
                    if (wide) {
                        swap_halves16(p);
                        if (r < rows) {
                            bf16_t* dst = orow + (c0 >> 1) + 16 * half;
                            *reinterpret_cast<u32x4*>(dst) = u32x4{p[0][0], p[0][1], p[2][0], p[2][1]};
                            *reinterpret_cast<u32x4*>(dst + 8) = u32x4{p[1][0], p[1][1], p[3][0], p[3][1]};
                        }
                    } else if (r < rows) {
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const int f = (c0 >> 1) + 8 * q + 4 * half;
#pragma unroll
                            for (int t = 0; t < 2; ++t) {
                                orow[f + 2 * t] = (bf16_t)(p[q][t] & 0xffff);
                                orow[f + 2 * t + 1] = (bf16_t)(p[q][t] >> 16);
                            }
                        }
                    }
                }
            }
        } else if constexpr (EPI == EPI_QKV) {
            static_assert(T::WM % 128 == 0, "a wave's rows must cover whole heads");
            if (a.head_dim == 128)
                qkv_epilogue<T::TM, T::TN, 128>(a, acc, m0, n0, lrow0, lcol0);
            else
                qkv_epilogue<T::TM, T::TN, 64>(a, acc, m0, n0, lrow0, lcol0);
        } else if constexpr (EPI == EPI_LMHEAD) {
            // rows = vocabulary ids, cols = tokens.  Per token: (max, first argmax,
            // sum exp(z - max)) over each half tile's BM/2 vocabulary rows.
            // Rows past the vocabulary exist only in the last tile: the checks
            // are compiled in for that tile alone (a wave-uniform branch).  The
            // exponent arguments are <= 0, so the hardware exp2 (no denormal
            // rescaling) serves; terms below 2^-126 of the maximum vanish.
            SoftmaxPartial part[T::TN];
            auto reduce = [&](auto checked) __attribute__((always_inline)) {
                constexpr bool CHK = decltype(checked)::value;
#pragma unroll
                for (int j = 0; j < T::TN; ++j) {
                    float m = -INFINITY;
                    int idx = 0x7fffffff;
#pragma unroll
                    for (int i = 0; i < T::TM; ++i)
#pragma unroll
                        for (int e = 0; e < 16; ++e) {
                            const int v = m0 + lrow0 + i * 32 + 8 * (e >> 2) + (e & 3);
                            const float z = (!CHK || v < rows) ? acc[i][j][e] : -INFINITY;
                            if (z > m) {
                                m = z;
                                idx = v;
                            }
                        }
                    float s = 0.f;
                    if (m != -INFINITY) {
                        const float ml = m * kLog2e;
#pragma unroll
                        for (int i = 0; i < T::TM; ++i)
#pragma unroll
                            for (int e = 0; e < 16; ++e) {
                                const int v = m0 + lrow0 + i * 32 + 8 * (e >> 2) + (e & 3);
                                if (!CHK || v < rows) s += __builtin_amdgcn_exp2f(acc[i][j][e] * kLog2e - ml);
                            }
                    }
                    // Merge with lane ^ 32 (the other half of the column's rows):
                    // v_permlane32_swap hands each lane its partner's values with
                    // no LDS round trip; lanes below 32 hold the lower rows.
                    const auto xm = __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false, false);
                    const auto xi = __builtin_amdgcn_permlane32_swap((uint32_t)idx, (uint32_t)idx, false, false);
                    const auto xs = __builtin_amdgcn_permlane32_swap(__float_as_uint(s), __float_as_uint(s), false, false);
                    const SoftmaxPartial lo{__uint_as_float(xm[0]), (int)xi[0], __uint_as_float(xs[0])};
                    const SoftmaxPartial hi{__uint_as_float(xm[1]), (int)xi[1], __uint_as_float(xs[1])};
                    part[j] = sp_merge(lo, hi);
                }
            };
            if (m0 + BM <= rows)
                reduce(std::false_type{});
            else
                reduce(std::true_type{});
            // One partial per (BM/2-row half tile, token): the two wave rows
            // (wm = 0, 1) write separately and the merge kernel combines them.
            if (lane < 32) {
                const int half = (m0 / BM) * 2 + wm;
#pragma unroll
                for (int j = 0; j < T::TN; ++j) {
                    const int c = n0 + lcol0 + j * 32;
                    if (c < a.N)
                        a.partials[(int64_t)half * a.N + c] =
                            make_float4(part[j].m, __int_as_float(part[j].idx), part[j].s, 0.f);
                }
            }
        }
    };

    // Software pipeline over K tiles (A of tile kt lives in A stage kt % SA,
    // B in B stage kt % SB;
    // registers hold every fragment of the tile being multiplied).  Per tile,
    // in phases the compiler may not reorder across:
    //   [steps 0 .. PRE-1 of tile kt ran at the end of the previous tile]
    //   wait until this wave's copy of tile kt+1 landed (its reads of tile kt
    //   finished long ago); barrier: tile kt+1 is complete in LDS and the
    //   stage of tile kt is free;
    //   step PRE      | copies of A tile kt+SA and B tile kt+SB into the freed stages
    //                 | reads of tile kt+1 slots 0 .. PRE-1 (their steps are done)
    //   step s > PRE  | reads of slot s-1
    //   step 0 of kt+1 | reads of slot KS-1
    //   steps 1 .. PRE-1 of kt+1
    // so every read has at least one phase of MFMAs to land before its use or
    // the next barrier.  Copies are always issued (clamped to the last tile
    // past the end of K, into a stage that is never multiplied), which keeps
    // every wait count a compile-time constant.
    const int nk = a.K / BK;
    // With more K tiles than stages, copies run continuously across tiles:
    // once a tile's own copies are all issued, the copy slots of its last
    // iterations fetch the next tile's first K tiles (stage indices carry
    // over), so a tile switch leaves one round of copies and no drain.
    // Otherwise every tile starts from a prologue of its own.
    const bool cont = nk > T::SD;
    if constexpr (PP) {
        // Ping-pong schedule (8 waves, two per SIMD).  Waves 0-3 (group 0, the
        // first BM/2 rows of the tile) and waves 4-7 (group 1, the other half)
        // alternate between a compute phase (all MFMAs of one K tile and nothing
        // else) and a memory phase (one round of copies into LDS, then every
        // fragment of the next K tile read into registers); a workgroup barrier
        // ends each phase.  While one wave of a SIMD multiplies, the other loads,
        // so the matrix core is never left waiting on LDS or on the other wave.
        // K tile k is read by group 0 in phase 2k and by group 1 in phase 2k+1,
        // so its stages are free from phase 2k+2 on.  Group 0 copies the operand
        // with fewer stages (S = 2: issued in phase 2k+2 for K tile k+S, awaited
        // at the end of phase 2(k+S)-1), group 1 the one with more (S = 3: issued
        // in phase 2k+3, awaited at the end of its memory phase 2(k+S)-1).  In
        // both cases S-2 later rounds of the same wave may still be in flight at
        // the wait.  Output tiles follow each other without a drain (as in the
        // other schedule): a group stores a finished tile at the start of its
        // next memory phase.
        static_assert(NW == 8 && T::SS == 2 && T::SD == 3, "ping-pong: 8 waves, 2 + 3 stages");
        auto group = [&](auto gc) __attribute__((always_inline)) {
            constexpr int G = decltype(gc)::value;
            constexpr int S = G == 0 ? T::SS : T::SD;                // stages of the operand this group copies
            constexpr bool CA = (G == 0) == (SA <= SB);               // this group copies A (else B)
            constexpr int OP_BYTES = CA ? T::A_BYTES : T::B_BYTES;
            constexpr int NI = OP_BYTES / 1024 / (NW / 2);             // 1 KB copy blocks per wave and K tile
            constexpr int OP_BASE = CA ? 0 : B_BASE;
            const int gw = wn;                                          // wave within the group
            buf_rsrc_t rsrc;
            uint32_t off[NI];
            auto setup = [&](const TileIdx& t) __attribute__((always_inline)) {
                // Lane terms recomputed from an opaque copy of the lane id, so
                // that they are not kept live across the K loop.
                int ln = lane;
                asm volatile("" : "+v"(ln));
                const int rin = ln / CPR, pc = ln % CPR;
                if constexpr (CA) {
                    rsrc = make_rsrc(gather ? a.A : a.A + (int64_t)(t.row_base + t.m0) * a.lda);
#pragma unroll
                    for (int p = 0; p < NI; ++p) {
                        const int tr = (gw * NI + p) * RPB + rin;
                        const int r = min(t.m0 + tr, t.rows - 1);
                        const int64_t grow = gather ? (int64_t)a.a_rows[t.row_base + r] : (int64_t)(r - t.m0);
                        off[p] = (uint32_t)(grow * a.lda * 2) + (uint32_t)((pc ^ swz_key<CPR>(tr)) * 16);
                    }
                } else {
                    const bf16_t* Bg = a.B + (GROUPED ? (int64_t)t.g * a.b_group_stride : 0);
                    rsrc = make_rsrc(Bg + (int64_t)t.n0 * a.ldb);
#pragma unroll
                    for (int p = 0; p < NI; ++p) {
                        const int tr = (gw * NI + p) * RPB + rin;
                        const int n = min(t.n0 + tr, a.N - 1) - t.n0;
                        off[p] = (uint32_t)((int64_t)n * a.ldb * 2) + (uint32_t)((pc ^ swz_key<CPR>(tr)) * 16);
                    }
                }
            };
            auto copy = [&](int kt, int stage) {                       // this group's part of K tile kt
                const int dst = OP_BASE + stage * OP_BYTES + gw * NI * 1024;
#pragma unroll
                for (int p = 0; p < NI; ++p) lds_dma16_buf(rsrc, off[p], kt * (BK * 2), lds_at(dst + p * 1024));
            };
            auto start = [&](const TileIdx& t) {                       // K tiles 0 .. S-1 into stages 0 .. S-1
                setup(t);
#pragma unroll
                for (int s = 0; s < S; ++s) copy(min(s, nk - 1), s);
            };
            // All MFMAs of one K tile.  The first K tile of an output tile
            // starts from a zero accumulator (an inline-constant operand), so
            // the accumulators are never cleared separately; it is multiplied
            // even by a wave with no rows in the tile, which keeps no older
            // accumulator live.
            auto compute = [&](auto first_tag) __attribute__((always_inline)) {
                constexpr bool FIRST = decltype(first_tag)::value;
#pragma unroll
                for (int ks = 0; ks < T::KS; ++ks)
#pragma unroll
                    for (int i = 0; i < T::TM; ++i)
#pragma unroll
                        for (int j = 0; j < T::TN; ++j) {
                            const f32x16 c = (FIRST && ks == 0) ? f32x16{} : acc[i][j];
                            acc[i][j] = TACC ? mfma32x32x16(rb[ks][j], ra[ks][i], c)
                                             : mfma32x32x16(ra[ks][i], rb[ks][j], c);
                        }
            };
            // A wave whose rows all lie past the end of a grouped tile's rows
            // skips its MFMAs but still copies, reads and meets every barrier.
            auto active = [&](const TileIdx& t) { return !GROUPED || t.m0 + wm * T::WM < t.rows; };

            TileIdx cur = decode(L), prv = cur;
            bool act = active(cur);
            bool pend = false;                  // tile prv awaits its epilogue (stored in K step 0)
            int sa = 0, sb = 0;                 // stages of the next K tile to read
            bool fresh = true;                  // the current tile began with a prologue
            start(cur);
            wait_vmcnt<NI * (S - 1)>();         // own part of K tile 0 landed
            lds_barrier();
            if constexpr (G == 1) lds_barrier();     // phase 0: group 0 reads, group 1 waits
            while (true) {
                const int L_next = L + stride;
                const bool more = L_next < x_end;
                const TileIdx nxt = more ? decode(L_next) : cur;
                const bool flow = cont && more;
                // One K tile: copy local K tile x (x < 0: none) into the stage
                // of K tile kt-1, read K tile kt, barrier, multiply, barrier.
                // K step 0 of a tile that follows another without a drain also
                // stores that tile in its memory phase: a store-only epilogue
                // after the copy (and, for group 1, after its wait, so that the
                // stores are newer than every copy awaited before the next
                // phase), one that also loads before the copy.
                constexpr bool EPI_LOADS = EPI == EPI_RESID || EPI == EPI_QKV;
                auto step = [&](int kt, int x, auto first_tag) __attribute__((always_inline)) {
                    constexpr bool FIRST = decltype(first_tag)::value;
                    // ---- memory phase
                    const int so = CA ? sa : sb;                        // own stage of K tile kt
                    bool waited = false;
                    if constexpr (FIRST && EPI_LOADS) {
                        // An epilogue that loads must not wait behind this
                        // phase's copies: it runs before them.
                        if (pend) {
                            epilogue(prv.m0, prv.rows, prv.row_base, prv.n0);
                            sched_fence();
                            pend = false;
                        }
                    }
                    if (x >= 0) copy(x, so == 0 ? S - 1 : so - 1);
                    if constexpr (FIRST && !EPI_LOADS) {
                        if (pend) {
                            if constexpr (G == 1) wait_vmcnt<NI * (S - 2)>();   // own part of K tile 1 landed
                            sched_fence();
                            epilogue(prv.m0, prv.rows, prv.row_base, prv.n0);
                            sched_fence();
                            pend = false;
                            waited = true;
                        }
                    }
                    set_stage(sa, sb);
#pragma unroll
                    for (int ks = 0; ks < T::KS; ++ks) read_slot(ks);
                    sa = sa + 1 == SA ? 0 : sa + 1;
                    sb = sb + 1 == SB ? 0 : sb + 1;
                    if constexpr (G == 1) {
                        if (!waited) wait_vmcnt<NI * (S - 2)>();        // own part of K tile kt+1 landed
                    }
                    sched_fence();
                    lds_barrier();
                    // ---- compute phase
                    if (FIRST || act) compute(first_tag);
                    sched_fence();
                    if constexpr (G == 0) wait_vmcnt<NI * (S - 2)>();   // own part of K tile kt+1 landed
                    lds_barrier();
                    sched_fence();
                };
                // Copies issued in K step kt fetch K tile kt-1+S.  With
                // continuous copies, those past the end fetch the next tile's
                // first K tiles (its offsets are set up between the two loops);
                // otherwise they repeat the last K tile into a stage that is
                // never read, which keeps every wait count constant.
                const int kt_sw = flow ? nk + 1 - S : nk;
                step(0, fresh ? -1 : min(S - 1, nk - 1), std::true_type());
                for (int kt = 1; kt < kt_sw; ++kt) step(kt, min(kt - 1 + S, nk - 1), std::false_type());
                if (flow) {
                    setup(nxt);
#pragma unroll
                    for (int c = 0; c < S - 1; ++c) step(kt_sw + c, c, std::false_type());
                    prv = cur;
                    pend = true;
                    cur = nxt;
                    L = L_next;
                    act = active(cur);
                    fresh = false;
                    continue;
                }
                // Drain: group 0 stores while group 1 multiplies its last K
                // tile (one more barrier for group 0), then group 1 stores.
                epilogue(cur.m0, cur.rows, cur.row_base, cur.n0);
                if constexpr (G == 0) __syncthreads();
                if (!more) break;
                // Short K (no continuous copies): every copy lands before the
                // next tile's prologue refills the stages.
                wait_all_memory();
                __syncthreads();
                cur = nxt;
                L = L_next;
                act = active(cur);
                sa = sb = 0;
                fresh = true;
                start(cur);
                wait_vmcnt<NI * (S - 1)>();
                lds_barrier();
                if constexpr (G == 1) lds_barrier();
            }
        };
        if (wm == 0) group(std::integral_constant<int, 0>());
        else group(std::integral_constant<int, 1>());
    } else {
    TileIdx cur = decode(L);
    setup_a(cur);
    setup_b(cur);
    prologue(nk);
    int sa0 = 0, sb0 = 0;                   // stages of K tile 0 of the current tile
    bool first = true;

    // ---------------------------------------------------------------- per tile
    while (true) {
    const int m0 = cur.m0, rows = cur.rows, row_base = cur.row_base, n0 = cur.n0;
    const int L_next = L + stride;
    const bool more = L_next < x_end;
    const TileIdx nxt = more ? decode(L_next) : cur;
    const bool flow = cont && more;          // this tile's loop also copies for the next tile
#pragma unroll
    for (int i = 0; i < T::TM; ++i)
#pragma unroll
        for (int j = 0; j < T::TN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
    if (first || !cont) wait_vmcnt<T::N_TOP>();   // K tile 0 landed, later ones may fly
    else wait_vmcnt<T::N_LOOP>();                 // the continuous pipeline's steady-state wait
    __syncthreads();
    // In grouped mode the last row tile of a group is often partly empty; a
    // wave whose rows all lie past the group's end skips its MFMAs (and
    // fragment reads) but still copies and meets every barrier.
    auto run = [&](auto active) {
        constexpr bool ACTIVE = decltype(active)::value;
        set_stage(sa0, sb0);
        if constexpr (ACTIVE) {
#pragma unroll
            for (int ks = 0; ks < T::KS; ++ks) read_slot(ks);
#pragma unroll
            for (int ks = 0; ks < PRE; ++ks) mfmas(ks);
        }
        sched_fence();

        int sa = sa0, sb = sb0;                 // stages of K tile kt
        for (int kt = 0; kt < nk - 1; ++kt) {
            const int na = sa + 1 == SA ? 0 : sa + 1, nb = sb + 1 == SB ? 0 : sb + 1;
            wait_vmcnt<T::N_LOOP>();                                // own copies of tile kt+1 landed
            __syncthreads();
            set_stage(na, nb);
            // Copies of K tiles kt+SA / kt+SB: past the end they belong to the
            // next tile, whose offsets replace this tile's once its last own
            // copy is out (set up here, where fragment slots 0 .. PRE-1 are free).
            int ka = kt + SA, kb = kt + SB;
            if (flow) {
                // The indices pass through an empty asm so that the offset
                // arithmetic is done here, not hoisted out of the K loop (where
                // its registers would stay live for the whole tile).
                TileIdx t = nxt;
                asm volatile("" : "+s"(t.g), "+s"(t.m0), "+s"(t.row_base), "+s"(t.rows), "+s"(t.n0));
                if (ka == nk) setup_a(t);
                if (kb == nk) setup_b(t);
                if (ka >= nk) ka -= nk;
                if (kb >= nk) kb -= nk;
            } else {
                ka = min(ka, nk - 1);
                kb = min(kb, nk - 1);
            }
            sched_fence();
            // step PRE | the copies | reads of slots 0 .. PRE-1 of tile kt+1
            if constexpr (ACTIVE) mfmas(PRE);
            issue(ka, sa, kb, sb);
            if constexpr (!ACTIVE) {
                sa = na;
                sb = nb;
                continue;
            }
#pragma unroll
            for (int q = 0; q < PRE; ++q) read_slot(q);
            constexpr int NRD = PRE * NR;
#pragma unroll
            for (int r = 0; r < NM; ++r) {
                sched_group<0x008, 1>();
#pragma unroll
                for (int c = r * (T::A_INSTR + T::B_INSTR) / NM; c < (r + 1) * (T::A_INSTR + T::B_INSTR) / NM; ++c)
                    sched_group<0x020, 1>();
#pragma unroll
                for (int c = r * NRD / NM; c < (r + 1) * NRD / NM; ++c) sched_group<0x100, 1>();
            }
            sched_fence();
#pragma unroll
            for (int ks = PRE + 1; ks < T::KS; ++ks) {                // step ks | reads of slot ks-1
                mfmas(ks);
                read_slot(ks - 1);
#pragma unroll
                for (int r = 0; r < NM; ++r) {
                    sched_group<0x008, 1>();
#pragma unroll
                    for (int c = r * NR / NM; c < (r + 1) * NR / NM; ++c) sched_group<0x100, 1>();
                }
                sched_fence();
            }
            mfmas(0);                                                 // step 0 of tile kt+1 | last slot
            read_slot(T::KS - 1);
#pragma unroll
            for (int r = 0; r < NM; ++r) {
                sched_group<0x008, 1>();
#pragma unroll
                for (int c = r * NR / NM; c < (r + 1) * NR / NM; ++c) sched_group<0x100, 1>();
            }
            sched_fence();
#pragma unroll
            for (int ks = 1; ks < PRE; ++ks) mfmas(ks);
            sched_fence();
            sa = na;
            sb = nb;
        }
        if constexpr (ACTIVE) {
#pragma unroll
            for (int ks = PRE; ks < T::KS; ++ks) mfmas(ks);         // last tile
        }
    };
    if (!GROUPED || m0 + wm * T::WM < rows) run(std::true_type());
    else run(std::false_type());
    if (flow) {
        // Every wave is done reading K tile nk-1: its stages take the last
        // round of the next tile's first copies (A tile SA-1, B tile SB-1).
        __syncthreads();
        issue(SA - 1, (sa0 + nk - 1) % SA, SB - 1, (sb0 + nk - 1) % SB);
        sa0 = (sa0 + nk) % SA;
        sb0 = (sb0 + nk) % SB;
    } else {
        // No copy may still be in flight into LDS when the workgroup moves on
        // (or ends); the next tile, if any, starts from its own prologue.
        wait_all_memory();
        __syncthreads();
        if (more) {
            setup_a(nxt);
            setup_b(nxt);
            prologue(nk);
            sa0 = sb0 = 0;
        }
    }

    epilogue(m0, rows, row_base, n0);
    if (!more) break;
    cur = nxt;
    L = L_next;
    first = false;
    }
    }
}

template <int BM, int BN, int BK, int SA, int SB, int NW, int EPI, bool GROUPED, bool PP>
hipError_t launch_t(const GemmArgs& a, int max_tiles, hipStream_t st) {
    if constexpr (EPI == EPI_QKV && (BM / 2) % 128 != 0) {
        return hipErrorInvalidValue;                       // RoPE pairs must stay inside one wave
    } else {
    auto kernel = gemm_kernel<BM, BN, BK, SA, SB, NW, EPI, GROUPED, PP>;
    // Workgroups that fit on the device at once (a multiple of 8, one share
    // per XCD), cached per device for this kernel; a persistent grid of at
    // most that many walks all tiles.  Concurrent first calls compute the same
    // value, so the relaxed atomic cache is race-free.
    static std::atomic<int> resident_of[kMaxDevices];
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    int resident = resident_of[dev].load(std::memory_order_relaxed);
    if (resident == 0) {
        int cus = 0, occ = 0;
        e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        if (e == hipSuccess) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kernel, NW * 64, 0);
        if (e != hipSuccess) return e;
        resident = std::max(8, cus * std::max(occ, 1) / 8 * 8);
        resident_of[dev].store(resident, std::memory_order_relaxed);
    }
    const int tiles_n = (a.N + BN - 1) / BN;
    const int tiles_m = GROUPED ? max_tiles : (a.M + BM - 1) / BM;
    int64_t blocks = (int64_t)tiles_m * tiles_n;
    if (blocks <= 0) return hipSuccess;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    blocks = std::min<int64_t>((blocks + 7) / 8 * 8, resident);
    hipLaunchKernelGGL(kernel, dim3((unsigned)blocks), dim3(NW * 64), 0, st, a);
    return hipGetLastError();
    }
}

// Tile configurations: BM x BN x BK, SA / SB LDS stages for A / B, NW waves.
// variant 0: 4 waves; 1: alternative stage/BK choices; 2: 8 waves, 2+2
// stages; 5: 8 waves with a third B stage (B streamed from far memory, e.g.
// expert weights); 6: 8 waves with a third A stage (A streamed, e.g. the LM
// head's vocabulary rows); 11 / 12: as 5 / 6 with the ping-pong schedule (the
// two waves of a SIMD alternate between multiplying and loading).  The
// 256x256 8-wave tiles with a third stage use all 160 KB of LDS.
template <int EPI, bool GROUPED>
hipError_t launch_tiles(const GemmArgs& a, int bm, int bn, int max_tiles, hipStream_t st) {
    if (a.variant == 1) {
        if (bm == 256 && bn == 256) return launch_t<256, 256, 32, 4, 4, 4, EPI, GROUPED, false>(a, max_tiles, st);
        if (bm == 128 && bn == 128) return launch_t<128, 128, 64, 3, 3, 4, EPI, GROUPED, false>(a, max_tiles, st);
        if (bm == 256 && bn == 128) return launch_t<256, 128, 64, 2, 2, 4, EPI, GROUPED, false>(a, max_tiles, st);
        return hipErrorInvalidValue;
    }
    if (bm == 256 && bn == 256) {
        if (a.variant == 2) return launch_t<256, 256, 64, 2, 2, 8, EPI, GROUPED, false>(a, max_tiles, st);
        if (a.variant == 5) return launch_t<256, 256, 64, 2, 3, 8, EPI, GROUPED, false>(a, max_tiles, st);
        if (a.variant == 6) return launch_t<256, 256, 64, 3, 2, 8, EPI, GROUPED, false>(a, max_tiles, st);
        if (a.variant == 11) return launch_t<256, 256, 64, 2, 3, 8, EPI, GROUPED, true>(a, max_tiles, st);
        if (a.variant == 12) return launch_t<256, 256, 64, 3, 2, 8, EPI, GROUPED, true>(a, max_tiles, st);
    }
    if (a.variant != 0) return hipErrorInvalidValue;
    if (bm == 256 && bn == 256) return launch_t<256, 256, 64, 2, 2, 4, EPI, GROUPED, false>(a, max_tiles, st);
    if (bm == 256 && bn == 128) return launch_t<256, 128, 64, 3, 3, 4, EPI, GROUPED, false>(a, max_tiles, st);
    if (bm == 128 && bn == 256) return launch_t<128, 256, 64, 3, 3, 4, EPI, GROUPED, false>(a, max_tiles, st);
    if (bm == 128 && bn == 128) return launch_t<128, 128, 64, 2, 2, 4, EPI, GROUPED, false>(a, max_tiles, st);
    if (bm == 128 && bn == 64) return launch_t<128, 64, 64, 2, 2, 4, EPI, GROUPED, false>(a, max_tiles, st);
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& a, int epi, bool grouped, int bm, int bn, int max_tiles,
                       hipStream_t st) {
    if (a.K % 64 != 0 || a.N <= 0 || (!grouped && a.M <= 0)) return hipErrorInvalidValue;
    switch (epi) {
        case EPI_BF16:
            return grouped ? launch_tiles<EPI_BF16, true>(a, bm, bn, max_tiles, st)
                           : launch_tiles<EPI_BF16, false>(a, bm, bn, max_tiles, st);
        case EPI_SWIGLU:
            return grouped ? launch_tiles<EPI_SWIGLU, true>(a, bm, bn, max_tiles, st)
                           : launch_tiles<EPI_SWIGLU, false>(a, bm, bn, max_tiles, st);
        case EPI_F32:
            return grouped ? hipErrorInvalidValue : launch_tiles<EPI_F32, false>(a, bm, bn, max_tiles, st);
        case EPI_RESID:
            return grouped ? hipErrorInvalidValue : launch_tiles<EPI_RESID, false>(a, bm, bn, max_tiles, st);
        case EPI_QKV:
            return grouped ? hipErrorInvalidValue : launch_tiles<EPI_QKV, false>(a, bm, bn, max_tiles, st);
        case EPI_LMHEAD:
            return grouped ? hipErrorInvalidValue : launch_tiles<EPI_LMHEAD, false>(a, bm, bn, max_tiles, st);
        case EPI_F32_T:
            return grouped ? hipErrorInvalidValue : launch_tiles<EPI_F32_T, false>(a, bm, bn, max_tiles, st);
        default:
            return hipErrorInvalidValue;
    }
}
