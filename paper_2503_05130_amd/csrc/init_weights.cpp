// Host-side weight generation from the seeded random-init spec.
//
// Every element is an independent draw: two outputs of the SplitMix64 output
// function (Steele, Lea & Flood, OOPSLA 2014) keyed by (seed, tensor uid,
// element index), turned into one standard normal by the Box-Muller transform
// (Box & Muller, 1958), scaled, then rounded fp64 -> fp32 -> bf16 with round to
// nearest even.  Counter-based, so any element can be produced independently
// and the work splits over threads without changing a single bit.  Generated
// on the host (glibc libm) -- never on the device, whose math library differs.
#include "init_weights.h"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <thread>
#include <vector>

namespace iefwd {

namespace {

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;

inline uint64_t splitmix_output(uint64_t s) {
    uint64_t z = s + kGolden;
    z ^= z >> 30;
    z *= 0xBF58476D1CE4E5B9ull;
    z ^= z >> 27;
    z *= 0x94D049BB133111EBull;
    z ^= z >> 31;
    return z;
}

inline double normal_draw(uint64_t key, uint64_t index) {
    const uint64_t c = key + (index << 1);
    const uint64_t r1 = splitmix_output(c);
    const uint64_t r2 = splitmix_output(c + 1);
    const double u1 = std::ldexp((double)((r1 >> 11) + 1), -53);   // (0, 1]
    const double u2 = std::ldexp((double)(r2 >> 11), -53);         // [0, 1)
    const double radius = std::sqrt(-2.0 * std::log(u1));
    const double angle = 6.283185307179586 * u2;
    return radius * std::cos(angle);
}

inline uint16_t bf16_rne(float f) {
    uint32_t u;
    std::memcpy(&u, &f, sizeof u);
    const uint32_t rounding = 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)((u + rounding) >> 16);
}

// Runs fn(begin, end) over [0, n) on up to hardware_concurrency threads.
template <class Fn>
void parallel_range(uint64_t n, Fn fn) {
    unsigned nt = std::max(1u, std::thread::hardware_concurrency());
    nt = (unsigned)std::min<uint64_t>(nt, std::max<uint64_t>(1, n / 65536));
    if (nt <= 1) {
        fn(0, n);
        return;
    }
    std::vector<std::thread> pool;
    pool.reserve(nt);
    const uint64_t step = (n + nt - 1) / nt;
    for (unsigned t = 0; t < nt; ++t) {
        const uint64_t b = t * step, e = std::min(n, b + step);
        if (b >= e) break;
        pool.emplace_back([=] { fn(b, e); });
    }
    for (auto &th : pool) th.join();
}

}  // namespace

uint64_t tensor_key(uint64_t seed, uint32_t layer, uint32_t slot) {
    const uint64_t uid = (uint64_t)layer * 32u + slot;
    return splitmix_output(seed ^ splitmix_output(uid));
}

void generate_matrix_transposed(uint64_t key, uint32_t in_dim, uint32_t out_dim, uint32_t qk_cols,
                                double sigma, double sigma_qk, uint16_t *dst) {
    // logical element e = i * out_dim + o (row-major [in, out]) lands at
    // dst[o * in_dim + i] (row-major [out, in])
    const bool split = sigma_qk != 0.0 && qk_cols > 0;
    parallel_range(out_dim, [&](uint64_t o0, uint64_t o1) {
        for (uint64_t o = o0; o < o1; ++o) {
            const double s = (split && o < qk_cols) ? sigma_qk : sigma;
            uint16_t *row = dst + o * in_dim;
            for (uint64_t i = 0; i < in_dim; ++i) {
                const float v = (float)(s * normal_draw(key, i * out_dim + o));
                row[i] = bf16_rne(v);
            }
        }
    });
}

void generate_vector_bf16(uint64_t key, uint32_t n, double sigma, uint16_t *dst) {
    for (uint32_t e = 0; e < n; ++e) dst[e] = bf16_rne((float)(sigma * normal_draw(key, e)));
}

void generate_vector_f32(uint64_t key, uint32_t n, double offset, double sigma, float *dst) {
    for (uint32_t e = 0; e < n; ++e) {
        const double scaled = sigma * normal_draw(key, e);
        dst[e] = (float)(offset + scaled);
    }
}

}  // namespace iefwd
