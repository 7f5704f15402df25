/*
 * Oracle weight generator -- TEST INFRASTRUCTURE ONLY.
 *
 * Part of the CPU oracle that checks the GPU library.  Only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg may load it; the
 * product path never does.  It shares no code, header or constant table
 * with the GPU library: both sides implement the same two published
 * algorithms independently, and a test compares their outputs bit for bit.
 *
 * Algorithms:
 *   Philox4x32-10: Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers:
 *   As Easy as 1, 2, 3" (SC'11).  A round maps counter (c0,c1,c2,c3) with
 *   key (k0,k1) to (hi(M1*c2)^c1^k0, lo(M1*c2), hi(M0*c0)^c3^k1, lo(M0*c0))
 *   with M0 = 0xD2511F53, M1 = 0xCD9E8D57; between rounds the key is bumped
 *   by the Weyl constants (0x9E3779B9, 0xBB67AE85).  Ten rounds.
 *   Box-Muller (1958): u1,u2 uniform in (0,1) give
 *   z0 = sqrt(-2 ln u1) cos(2 pi u2), z1 = sqrt(-2 ln u1) sin(2 pi u2).
 *
 * Weight rule (random-init policy weights, N(0, std)): element i of a tensor
 * (row-major in its logical [out, in] layout) belongs to pair j = i / 2.
 * Philox key = (lo32(seed), hi32(seed)); counter = (lo32(j), hi32(j),
 * tensor_id, 0).  Outputs x0, x1 give u = (x + 0.5) * 2^-32 in double,
 * Box-Muller gives z0 (even element) and z1 (odd element), and the weight
 * is (float)(std * z), then rounded to bfloat16 (nearest-even) for bf16
 * models.  All arithmetic in double with the C library's log/cos/sin.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

static void philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4])
{
    uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)c0;
        uint64_t p1 = (uint64_t)0xCD9E8D57u * (uint64_t)c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        uint32_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Raw generator output, exposed so tests can check the u32 stream itself. */
void orc_philox(uint64_t seed, const uint32_t ctr[4], uint32_t out[4])
{
    uint32_t key[2] = { (uint32_t)seed, (uint32_t)(seed >> 32) };
    philox4x32_10(ctr, key, out);
}

static uint16_t f32_to_bf16_rne(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    uint32_t lsb = (u >> 16) & 1u;
    u += 0x7FFFu + lsb;
    return (uint16_t)(u >> 16);
}

/* One Box-Muller pair from one Philox draw. */
static void normal_pair(uint64_t seed, uint32_t tensor_id, uint64_t j, double out[2])
{
    uint32_t ctr[4] = { (uint32_t)j, (uint32_t)(j >> 32), tensor_id, 0u };
    uint32_t x[4];
    orc_philox(seed, ctr, x);
    const double two_pow_m32 = 1.0 / 4294967296.0;
    double u1 = ((double)x[0] + 0.5) * two_pow_m32;
    double u2 = ((double)x[1] + 0.5) * two_pow_m32;
    double r = sqrt(-2.0 * log(u1));
    double t = 6.283185307179586 * u2;
    out[0] = r * cos(t);
    out[1] = r * sin(t);
}

/* Fill `count` fp32 weights N(0, stdv) of tensor `tensor_id`. */
void orc_normal_f32(uint64_t seed, uint32_t tensor_id, int64_t count, double stdv, float* out)
{
    int64_t pairs = (count + 1) / 2;
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < pairs; ++j) {
        double z[2];
        normal_pair(seed, tensor_id, (uint64_t)j, z);
        for (int h = 0; h < 2; ++h) {
            int64_t i = 2 * j + h;
            if (i < count) out[i] = (float)(stdv * z[h]);
        }
    }
}

/* Same values, rounded once more to bfloat16 (raw 16-bit patterns). */
void orc_normal_bf16(uint64_t seed, uint32_t tensor_id, int64_t count, double stdv, uint16_t* out)
{
    int64_t pairs = (count + 1) / 2;
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < pairs; ++j) {
        double z[2];
        normal_pair(seed, tensor_id, (uint64_t)j, z);
        for (int h = 0; h < 2; ++h) {
            int64_t i = 2 * j + h;
            if (i < count) out[i] = f32_to_bf16_rne((float)(stdv * z[h]));
        }
    }
}
