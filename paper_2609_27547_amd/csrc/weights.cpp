// Seeded random-init weights of the policy (host side).
//
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of
//   (c0, c1, c2, c3) <- (mulhi(B, c2) ^ c1 ^ k0, mullo(B, c2),
//                        mulhi(A, c0) ^ c3 ^ k1, mullo(A, c0))
// with A = 0xD2511F53, B = 0xCD9E8D57 and the key advanced by
// (0x9E3779B9, 0xBB67AE85) before every round but the first.
// Each pair of consecutive elements of a tensor (logical [out, in]
// row-major order) takes one draw: counter (lo(j), hi(j), tensor id, 0),
// key (lo(seed), hi(seed)); the first two words become u = (x + 1/2) 2^-32
// and a Box-Muller transform (1958) gives two standard normals, scaled by
// the init std in double and rounded to float (then to bf16, nearest even,
// for bf16 policies).
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <thread>
#include <vector>

#include "weights.h"

namespace ebrl {

static inline void philox10(uint32_t c[4], uint32_t k0, uint32_t k1) {
    for (int r = 0; r < 10; ++r) {
        if (r) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        const uint64_t pa = 0xD2511F53ull * c[0];
        const uint64_t pb = 0xCD9E8D57ull * c[2];
        const uint32_t n0 = (uint32_t)(pb >> 32) ^ c[1] ^ k0;
        const uint32_t n2 = (uint32_t)(pa >> 32) ^ c[3] ^ k1;
        c[1] = (uint32_t)pb;
        c[3] = (uint32_t)pa;
        c[0] = n0;
        c[2] = n2;
    }
}

static inline uint16_t round_bf16(float f) {
    uint32_t u;
    memcpy(&u, &f, sizeof(u));
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

static void gen_range(uint64_t seed, uint32_t tid, int64_t count, double stdv, bool bf16, void* out,
                      int64_t pair_lo, int64_t pair_hi) {
    const uint32_t k0 = (uint32_t)(seed & 0xFFFFFFFFu), k1 = (uint32_t)(seed >> 32);
    const double scale32 = 1.0 / 4294967296.0;
    for (int64_t j = pair_lo; j < pair_hi; ++j) {
        uint32_t c[4] = {(uint32_t)((uint64_t)j & 0xFFFFFFFFu), (uint32_t)((uint64_t)j >> 32), tid, 0u};
        philox10(c, k0, k1);
        const double u1 = ((double)c[0] + 0.5) * scale32;
        const double u2 = ((double)c[1] + 0.5) * scale32;
        const double rad = sqrt(-2.0 * log(u1));
        const double ang = 6.283185307179586 * u2;
        const double z[2] = {rad * cos(ang), rad * sin(ang)};
        for (int h = 0; h < 2; ++h) {
            const int64_t e = 2 * j + h;
            if (e >= count) break;
            const float w = (float)(stdv * z[h]);
            if (bf16) static_cast<uint16_t*>(out)[e] = round_bf16(w);
            else static_cast<float*>(out)[e] = w;
        }
    }
}

void generate_weight(uint64_t seed, uint32_t tensor_id, int64_t count, double stdv, bool bf16,
                     void* out) {
    const int64_t pairs = (count + 1) / 2;
    unsigned nt = std::max(1u, std::thread::hardware_concurrency());
    nt = (unsigned)std::min<int64_t>(nt, std::max<int64_t>(1, pairs / 65536));
    if (nt <= 1) {
        gen_range(seed, tensor_id, count, stdv, bf16, out, 0, pairs);
        return;
    }
    std::vector<std::thread> th;
    const int64_t per = (pairs + nt - 1) / nt;
    for (unsigned t = 0; t < nt; ++t) {
        const int64_t lo = (int64_t)t * per, hi = std::min(pairs, lo + per);
        if (lo >= hi) break;
        th.emplace_back(gen_range, seed, tensor_id, count, stdv, bf16, out, lo, hi);
    }
    for (auto& x : th) x.join();
}

}  // namespace ebrl
