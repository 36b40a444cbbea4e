// Host-side checks of libiefwd's CPU code, built with AddressSanitizer and
// UndefinedBehaviorSanitizer (tests/test_host_sanitizers.py builds and runs
// it): the ABI's argument validation, the CU-mask builder, the quota
// controller and the seeded weight generator.  Every output buffer is a heap
// allocation of exactly the size the call may write, so an overrun is caught.
// No kernel is launched; instance creation either finds no device or is
// undone at once.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "iefwd.h"
#include "init_weights.h"

static int failures = 0;
#define CHECK(c)                                                              \
    do {                                                                      \
        if (!(c)) {                                                           \
            std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
            ++failures;                                                       \
        }                                                                     \
    } while (0)

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint64_t next_u64() {   // xorshift64*
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return rng_state * 2685821657736338717ull;
}
static double uniform() { return (double)(next_u64() >> 11) * (1.0 / 9007199254740992.0); }

static void check_configs() {
    iefwd_config base;
    iefwd_config_init(&base);   // defaults; the shape is the caller's
    base.n_layers = 1;
    base.d_model = 128;
    base.n_heads = 2;
    base.d_ff = 512;
    base.max_batch = 2;
    base.max_seq = 32;
    iefwd_instance *inst = reinterpret_cast<iefwd_instance *>(0x1);
    CHECK(iefwd_create(nullptr, 0, &inst) == IEFWD_EINVAL && inst == nullptr);
    CHECK(iefwd_create(&base, 0, nullptr) == IEFWD_EINVAL);
    struct Bad {
        const char *what;
        void (*edit)(iefwd_config &);
        int status;
    } bad[] = {
        {"abi_version", [](iefwd_config &c) { c.abi_version = 0; }, IEFWD_EVERSION},
        {"d_model 100", [](iefwd_config &c) { c.d_model = 100; }, IEFWD_EINVAL},
        {"d_model 8192", [](iefwd_config &c) { c.d_model = 8192; }, IEFWD_EINVAL},
        {"n_heads 0", [](iefwd_config &c) { c.n_heads = 0; }, IEFWD_EINVAL},
        {"head dim 96", [](iefwd_config &c) { c.d_model = 768; c.n_heads = 8; }, IEFWD_EINVAL},
        {"d_ff 63", [](iefwd_config &c) { c.d_ff = 63; }, IEFWD_EINVAL},
        {"n_layers 0", [](iefwd_config &c) { c.n_layers = 0; }, IEFWD_EINVAL},
        {"n_out 17", [](iefwd_config &c) { c.n_out = 17; }, IEFWD_EINVAL},
        {"max_batch 0", [](iefwd_config &c) { c.max_batch = 0; }, IEFWD_EINVAL},
        {"kv_cache 2", [](iefwd_config &c) { c.kv_cache = 2; }, IEFWD_EINVAL},
        {"kv_cache post-LN", [](iefwd_config &c) { c.kv_cache = 1; c.pre_ln = 0; c.causal = 1; }, IEFWD_EINVAL},
        {"ln_eps 0", [](iefwd_config &c) { c.ln_eps = 0.f; }, IEFWD_EINVAL},
        {"ln_eps NaN", [](iefwd_config &c) { c.ln_eps = std::nanf(""); }, IEFWD_EINVAL},
        {"w_std -1", [](iefwd_config &c) { c.w_std = -1.f; }, IEFWD_EINVAL},
        {"tokens too many", [](iefwd_config &c) { c.max_batch = 65535; c.max_seq = 65535; }, IEFWD_EINVAL},
    };
    for (const Bad &b : bad) {
        iefwd_config c = base;
        b.edit(c);
        inst = reinterpret_cast<iefwd_instance *>(0x1);
        const int st = iefwd_create(&c, 0, &inst);
        if (st != b.status) std::fprintf(stderr, "config %s: status %d\n", b.what, st);
        CHECK(st == b.status);
        CHECK(inst == nullptr);
        const char *msg = iefwd_last_error();
        CHECK(msg != nullptr && std::strlen(msg) > 0);
    }
    // a valid config: no device here (ENODEV); with one, the instance is destroyed at once
    inst = nullptr;
    const int st = iefwd_create(&base, 0, &inst);
    CHECK(st == IEFWD_OK || st == IEFWD_ENODEV);
    if (st == IEFWD_OK) CHECK(iefwd_destroy(inst) == IEFWD_OK);
    CHECK(iefwd_create(&base, -1, &inst) == IEFWD_ENODEV);
    for (int s = -8; s <= 1; ++s) CHECK(iefwd_status_string(s) != nullptr);
}

static void check_null_instance() {
    float f = 0.f;
    uint64_t u = 0;
    double d = 0.0;
    std::vector<float> x(16);
    CHECK(iefwd_submit(nullptr, x.data(), 1, 1, 0) == IEFWD_EINVAL);
    CHECK(iefwd_wait(nullptr) == IEFWD_EINVAL);
    CHECK(iefwd_set_quota(nullptr, 8) == IEFWD_EINVAL);
    CHECK(iefwd_set_quota_at(nullptr, 8, 0) == IEFWD_EINVAL);
    CHECK(iefwd_prepare_quota_at(nullptr, 8, 0) == IEFWD_EINVAL);
    CHECK(iefwd_set_stream_cache(nullptr, 2) == IEFWD_EINVAL);
    CHECK(iefwd_last_batch_ms(nullptr, &f) == IEFWD_EINVAL);
    CHECK(iefwd_kernels_launched(nullptr, &u) == IEFWD_EINVAL);
    CHECK(iefwd_kernel_time(nullptr, 0, &d, &u) == IEFWD_EINVAL);
    CHECK(iefwd_read_logits(nullptr, x.data(), x.size(), 0) == IEFWD_EINVAL);
    CHECK(iefwd_decode(nullptr, x.data(), 1, 0, 0) == IEFWD_EINVAL);
}

static void check_masks() {
    const uint32_t cus[] = {8, 16, 32, 40, 64, 96, 128, 200, 256, 304};
    const uint32_t xcds[] = {1, 2, 4, 8};
    for (uint32_t n_cu : cus)
        for (uint32_t n_xcd : xcds) {
            const uint32_t words = (n_cu + 31) / 32;
            for (int trial = 0; trial < 64; ++trial) {
                const uint32_t q = 1 + (uint32_t)(next_u64() % n_cu);
                const uint32_t first = (uint32_t)(next_u64() % n_cu);
                uint32_t *m = static_cast<uint32_t *>(std::malloc(words * sizeof(uint32_t)));
                const int st = iefwd_build_cu_mask(n_cu, n_xcd, q, first, m, words);
                if (n_cu % n_xcd) {
                    CHECK(st == IEFWD_EINVAL);
                } else {
                    CHECK(st == IEFWD_OK);
                    uint32_t bits = 0;
                    for (uint32_t w = 0; w < words; ++w) bits += (uint32_t)__builtin_popcount(m[w]);
                    CHECK(bits == q);
                    if (n_cu % 32) CHECK((m[words - 1] >> (n_cu % 32)) == 0);
                }
                std::free(m);
            }
            uint32_t *m = static_cast<uint32_t *>(std::malloc(words * sizeof(uint32_t)));
            CHECK(iefwd_build_cu_mask(n_cu, n_xcd, 0, 0, m, words) == IEFWD_EINVAL);
            CHECK(iefwd_build_cu_mask(n_cu, n_xcd, n_cu + 1, 0, m, words) == IEFWD_EINVAL);
            CHECK(iefwd_build_cu_mask(n_cu, n_xcd, 1, n_cu, m, words) == IEFWD_EINVAL);
            CHECK(iefwd_build_cu_mask(n_cu, 0, 1, 0, m, words) == IEFWD_EINVAL);
            if (words > 1) CHECK(iefwd_build_cu_mask(n_cu, n_xcd, 1, 0, m, words - 1) == IEFWD_EINVAL);
            CHECK(iefwd_build_cu_mask(n_cu, n_xcd, 1, 0, nullptr, words) == IEFWD_EINVAL);
            std::free(m);
        }
}

static void check_controller() {
    iefwd_ctl_params p;
    CHECK(iefwd_ctl_params_init(&p) == IEFWD_OK);
    iefwd_ctl *ctl = nullptr;
    iefwd_ctl_params bad = p;
    bad.granule = 0;
    CHECK(iefwd_ctl_create(&bad, &ctl) == IEFWD_EINVAL);
    bad = p;
    bad.min_quota = p.max_tokens + 1;
    CHECK(iefwd_ctl_create(&bad, &ctl) == IEFWD_EINVAL);
    bad = p;
    bad.eta_increase = 0.5;
    CHECK(iefwd_ctl_create(&bad, &ctl) == IEFWD_EINVAL);
    bad = p;
    bad.flags = 2;   // an undefined flag bit
    CHECK(iefwd_ctl_create(&bad, &ctl) == IEFWD_EINVAL);
    CHECK(iefwd_ctl_create(nullptr, &ctl) == IEFWD_EINVAL);
    CHECK(iefwd_ctl_destroy(nullptr) == IEFWD_OK);
    for (int stream = 0; stream < 40; ++stream) {
        iefwd_ctl_params q = p;
        q.max_tokens = 64u << (next_u64() % 3);   // 64, 128, 256
        q.granule = 1u << (next_u64() % 4);
        q.min_quota = q.granule * (1 + (uint32_t)(next_u64() % 2));
        q.window = 1 + (uint32_t)(next_u64() % 6);
        q.flags = (uint32_t)(next_u64() % 2) * IEFWD_CTL_TEMPORARY_YIELD;
        CHECK(iefwd_ctl_create(&q, &ctl) == IEFWD_OK);
        const uint32_t n = 1 + (uint32_t)(next_u64() % 6);
        for (uint32_t i = 0; i < n; ++i) {
            const double req = 0.05 + 0.45 * uniform();
            const double lim = req + (1.0 - req) * uniform();
            uint32_t id = 99;
            CHECK(iefwd_ctl_add(ctl, req, lim, (int)(next_u64() % 2), &id) == IEFWD_OK && id == i);
        }
        uint32_t id = 0;
        CHECK(iefwd_ctl_add(ctl, 0.6, 0.5, 0, &id) == IEFWD_EINVAL);   // request > limit
        CHECK(iefwd_ctl_report(ctl, n, 1, 1.0) == IEFWD_EINVAL);      // no such instance
        double *tokens = static_cast<double *>(std::malloc(n * sizeof(double)));
        uint32_t *quotas = static_cast<uint32_t *>(std::malloc(n * sizeof(uint32_t)));
        uint32_t *firsts = static_cast<uint32_t *>(std::malloc(n * sizeof(uint32_t)));
        CHECK(iefwd_ctl_issue(ctl, tokens, quotas, firsts, n + 1) == IEFWD_EINVAL);
        for (int period = 0; period < 300; ++period) {
            for (uint32_t i = 0; i < n; ++i) {
                if (next_u64() % 4 == 0) continue;                           // no report this period
                const uint64_t kernels = next_u64() % 3 == 0 ? 0 : next_u64() % 5000;
                const double klc = next_u64() % 5 == 0 ? 0.0 : 0.5 + 20.0 * uniform();
                CHECK(iefwd_ctl_report(ctl, i, kernels, klc) == IEFWD_OK);
            }
            const bool nulls = next_u64() % 8 == 0;
            CHECK(iefwd_ctl_issue(ctl, nulls ? nullptr : tokens, quotas, nulls ? nullptr : firsts, n) == IEFWD_OK);
            int32_t state = -1;
            CHECK(iefwd_ctl_state(ctl, &state) == IEFWD_OK && state >= 0 && state <= 3);
            for (uint32_t i = 0; i < n; ++i) {
                CHECK(quotas[i] >= q.min_quota && quotas[i] <= q.max_tokens);
                CHECK(quotas[i] % q.granule == 0 || quotas[i] == q.max_tokens);
                if (!nulls) {
                    CHECK(firsts[i] < q.max_tokens);
                    CHECK(std::isfinite(tokens[i]) && tokens[i] >= 0.0);
                }
            }
        }
        std::free(tokens);
        std::free(quotas);
        std::free(firsts);
        CHECK(iefwd_ctl_destroy(ctl) == IEFWD_OK);
    }
}

static void check_init() {
    const uint32_t shapes[][3] = {{128, 384, 256}, {768, 2304, 1536}, {1000, 7, 0}, {64, 4096, 0}};
    for (const auto &s : shapes) {
        const size_t n = (size_t)s[0] * s[1];
        uint16_t *a = static_cast<uint16_t *>(std::malloc(n * sizeof(uint16_t)));
        uint16_t *b = static_cast<uint16_t *>(std::malloc(n * sizeof(uint16_t)));
        const uint64_t key = iefwd::tensor_key(11, s[0], s[1] % 32);
        iefwd::generate_matrix_transposed(key, s[0], s[1], s[2], 0.02, 0.06, a);
        iefwd::generate_matrix_transposed(key, s[0], s[1], s[2], 0.02, 0.06, b);
        CHECK(std::memcmp(a, b, n * sizeof(uint16_t)) == 0);   // same key, same bits, any thread split
        size_t nonfinite = 0;
        for (size_t i = 0; i < n; ++i) nonfinite += (a[i] & 0x7f80u) == 0x7f80u;
        CHECK(nonfinite == 0);
        std::free(a);
        std::free(b);
    }
    const uint32_t lens[] = {1, 7, 768, 3072};
    for (uint32_t len : lens) {
        uint16_t *v = static_cast<uint16_t *>(std::malloc(len * sizeof(uint16_t)));
        float *g = static_cast<float *>(std::malloc(len * sizeof(float)));
        iefwd::generate_vector_bf16(iefwd::tensor_key(7, 0, 1), len, 0.02, v);
        iefwd::generate_vector_f32(iefwd::tensor_key(7, 0, 4), len, 1.0, 0.02, g);
        for (uint32_t i = 0; i < len; ++i) CHECK(std::isfinite(g[i]) && std::fabs(g[i] - 1.0f) < 0.5f);
        std::free(v);
        std::free(g);
    }
}

int main() {
    check_configs();
    check_null_instance();
    check_masks();
    check_controller();
    check_init();
    if (failures) {
        std::fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    std::printf("host sanitizer checks passed\n");
    return 0;
}
