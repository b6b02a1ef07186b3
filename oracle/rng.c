/*
 * CPU oracle -- test infrastructure only.  Only tests/, the smoke check and the
 * benchmark's CPU-baseline leg may load this library; the GPU product path
 * never does.
 *
 * Counter-based generator for the synthetic refiner weights, written from the
 * published definition of Philox4x32-10 (Salmon, Moraes, Dror, Shaw,
 * "Parallel random numbers: as easy as 1, 2, 3", SC'11): a 4x32-bit counter,
 * a 2x32-bit key, ten rounds of two 32x32->64 multiplies with the Philox
 * multipliers, key bumped by the Weyl constants between rounds.
 *
 * Synthetic weight element (shared definition, implemented separately on
 * each side):
 *   key     = (seed & 0xffffffff, seed >> 32)
 *   counter = (i & 0xffffffff, i >> 32, tensor_id, 0)
 *             with i the row-major element index of the logical
 *             [out_features x in_features] matrix
 *   (w0, w1, w2, w3) = Philox4x32-10(counter, key)
 *   n = lo16(w0) + hi16(w0) + lo16(w1) + hi16(w1) - 131070
 *       (an Irwin-Hall sum of four 16-bit uniforms, centred; |n| <= 131070)
 * The oracle returns n; scaling and bf16 rounding happen in weights.py.
 */
#include <stdint.h>

#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

void oracle_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
    uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += PHILOX_W0;
            k1 += PHILOX_W1;
        }
        uint64_t p0 = (uint64_t)PHILOX_M0 * (uint64_t)c0;
        uint64_t p1 = (uint64_t)PHILOX_M1 * (uint64_t)c2;
        uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
        uint32_t n1 = (uint32_t)p1;
        uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
        uint32_t n3 = (uint32_t)p0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Irwin-Hall integers n for elements [start, start+count) of one tensor. */
void oracle_irwin_hall(uint64_t seed, uint32_t tensor_id, uint64_t start, uint64_t count,
                       int32_t *out) {
    const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < (int64_t)count; ++j) {
        uint64_t i = start + (uint64_t)j;
        uint32_t ctr[4] = {(uint32_t)i, (uint32_t)(i >> 32), tensor_id, 0u};
        uint32_t w[4];
        oracle_philox4x32_10(ctr, key, w);
        int32_t s = (int32_t)(w[0] & 0xffffu) + (int32_t)(w[0] >> 16)
                  + (int32_t)(w[1] & 0xffffu) + (int32_t)(w[1] >> 16);
        out[j] = s - 131070;
    }
}

/* Same, for an arbitrary list of element indices (sampled checks). */
void oracle_irwin_hall_at(uint64_t seed, uint32_t tensor_id, const uint64_t *idx, uint64_t count,
                          int32_t *out) {
    const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < (int64_t)count; ++j) {
        uint64_t i = idx[j];
        uint32_t ctr[4] = {(uint32_t)i, (uint32_t)(i >> 32), tensor_id, 0u};
        uint32_t w[4];
        oracle_philox4x32_10(ctr, key, w);
        int32_t s = (int32_t)(w[0] & 0xffffu) + (int32_t)(w[0] >> 16)
                  + (int32_t)(w[1] & 0xffffu) + (int32_t)(w[1] >> 16);
        out[j] = s - 131070;
    }
}
