// libiefwd: C ABI, instances and the forward-pass executor.
//
// An instance is one serverless DL function instance in the paper's sense
// (Sec. 3.1 serving plane): its own model weights, its own workspace, and a
// compute share that the elasticity layer moves between a request and a limit
// at run time (Sec. 3.2, 3.4).  Each batch execution is one iteration; the
// share (a CU mask on the instance's stream) changes only between iterations.
#include "iefwd.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <memory>
#include <mutex>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "controller.h"
#include "init_weights.h"
#include "kernels.h"
#include "quota.h"

using namespace iefwd;

namespace iefwd {
LaunchEvents &armed_launch_events() {
    thread_local LaunchEvents ev;
    return ev;
}
uint64_t &launch_count() {
    thread_local uint64_t n = 0;
    return n;
}
}  // namespace iefwd

namespace {

thread_local std::string t_last_error;

struct Error {
    int status;
    std::string msg;
};

[[noreturn]] void fail(int status, const std::string &msg) { throw Error{status, msg}; }

void hip_check(hipError_t e, const char *what) {
    if (e != hipSuccess) fail(IEFWD_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

template <class F>
int guarded(F &&f) {
    t_last_error.clear();
    try {
        f();
        return IEFWD_OK;
    } catch (const Error &e) {
        t_last_error = e.msg;
        return e.status;
    } catch (const std::bad_alloc &) {
        t_last_error = "host allocation failed";
        return IEFWD_ENOMEM;
    } catch (...) {
        t_last_error = "unexpected internal error";
        return IEFWD_EHIP;
    }
}

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// ------------------------------------------------------------------------------- device

struct DeviceInfo {
    uint32_t n_cu, n_xcd;
};

DeviceInfo query_device(int device) {
    int count = 0;
    if (hipGetDeviceCount(&count) != hipSuccess || count <= 0) {
        (void)hipGetLastError();
        fail(IEFWD_ENODEV, "no HIP device available");
    }
    if (device < 0 || device >= count) fail(IEFWD_ENODEV, "device index out of range");
    hipDeviceProp_t prop;
    hip_check(hipGetDeviceProperties(&prop, device), "hipGetDeviceProperties");
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        fail(IEFWD_ENODEV, std::string("device is ") + prop.gcnArchName + ", not gfx950");
    int xcc = 0;
    if (hipDeviceGetAttribute(&xcc, hipDeviceAttributeNumberOfXccs, device) != hipSuccess || xcc <= 0) {
        (void)hipGetLastError();
        xcc = 8;
    }
    return DeviceInfo{(uint32_t)prop.multiProcessorCount, (uint32_t)xcc};
}

// ------------------------------------------------------------------------------- config

void validate_config(const iefwd_config &c) {
    if (c.abi_version != IEFWD_ABI_VERSION) fail(IEFWD_EVERSION, "config.abi_version mismatch");
    auto bad = [](const char *m) { fail(IEFWD_EINVAL, m); };
    if (c.kv_cache > 1) bad("kv_cache must be 0 or 1");
    if (c.kv_cache && !(c.pre_ln && c.causal)) bad("kv_cache (decode) needs pre_ln = 1 and causal = 1");
    if (c.kv_cache && c.max_seq > 8192) bad("kv_cache needs max_seq <= 8192");
    if (c.n_layers < 1 || c.n_layers > 4096) bad("n_layers must be in [1, 4096]");
    if (c.d_model < 128 || c.d_model > 4096 || c.d_model % 128 != 0) bad("d_model must be a multiple of 128 in [128, 4096]");
    if (c.n_heads < 1 || c.d_model % c.n_heads != 0) bad("n_heads must divide d_model");
    const uint32_t dh = c.d_model / c.n_heads;
    if (dh != 64 && dh != 128) bad("head dim d_model / n_heads must be 64 or 128");
    if (c.d_ff < 64 || c.d_ff > 65536 || c.d_ff % 64 != 0) bad("d_ff must be a multiple of 64 in [64, 65536]");
    if (c.n_out > 16) bad("n_out must be <= 16");
    if (c.pre_ln > 1 || c.causal > 1) bad("pre_ln and causal must be 0 or 1");
    if (c.max_batch < 1 || c.max_seq < 1) bad("max_batch and max_seq must be >= 1");
    if ((uint64_t)c.max_batch * c.n_heads > 65535) bad("max_batch * n_heads must be <= 65535");
    const uint64_t tmax = (uint64_t)c.max_batch * c.max_seq;
    // element offsets inside the GEMM are 32-bit: rows * K must stay below 2^31
    if (tmax * std::max<uint64_t>(c.d_ff, 3ull * c.d_model) >= (1ull << 31)) bad("max_batch * max_seq too large");
    if (!(c.ln_eps > 0.f) || !std::isfinite(c.ln_eps)) bad("ln_eps must be positive and finite");
    for (float s : {c.w_std, c.b_std, c.ln_std, c.qk_std})
        if (!(s >= 0.f) || !std::isfinite(s)) bad("init std values must be finite and >= 0");
}

// ------------------------------------------------------------------------------- instance

struct LayerWeights {
    bf16_t *wqkv, *bqkv, *wo, *bo, *w1, *b1, *w2, *b2;   // matrices output-major [out, in]
    float *g1, *be1, *g2, *be2;
    // decode instances: packed copies of wqkv, wo, w1, w2 for the skinny
    // product, and the K-group count each copy is packed for
    bf16_t *packed[4] = {nullptr, nullptr, nullptr, nullptr};
    int packed_groups[4] = {0, 0, 0, 0};
};

// Training state of an instance created with iefwd_train_create: the flat
// fp32 optimiser state (master weights, gradients, two moments, one segment
// per parameter tensor), transposed bf16 weights for the input-gradient
// products, the activations the forward saves per layer, and the backward's
// scratch.  One device allocation, carved.
struct TrainState {
    iefwd_train_params hp{};
    uint64_t steps = 0;
    void *blob = nullptr;
    float *loss_host = nullptr;                   // pinned: the last step's summed token losses
    // optimiser state, segments in (layer, slot) order then the head
    float *master = nullptr, *grad = nullptr, *mom1 = nullptr, *mom2 = nullptr;
    size_t n_params = 0;                          // padded element count
    std::vector<std::array<size_t, 12>> off;      // per layer: element offset of each slot
    size_t off_wh = 0, off_bh = 0;
    std::vector<AdamSegment> segs;
    AdamSegment *segs_d = nullptr;
    uint32_t *blk_seg_d = nullptr;
    int n_blocks = 0;
    // W^T [in, out] bf16 of the four matrices per layer
    struct Transposed {
        bf16_t *wqkv, *wo, *w1, *w2;
    };
    std::vector<Transposed> wt;
    // saved activations per layer (T = max_batch * max_seq rows)
    struct Saved {
        bf16_t *hb, *q, *k, *vt, *ctx, *h1b, *v, *u;
        float *z1, *st1, *z2, *st2;
    };
    std::vector<Saved> saved;
    // backward scratch
    float *dxa = nullptr, *dxb = nullptr, *dz = nullptr, *xl = nullptr, *loss_t = nullptr, *dlogits = nullptr;
    float *colpart = nullptr, *loss_sum = nullptr;   // column-sum partials of one layer; the loss
    bf16_t *dzb = nullptr, *dvb = nullptr, *dctx = nullptr, *dqkv = nullptr, *ta = nullptr, *tb = nullptr;
    bf16_t *zero_bias = nullptr, *attn_scratch = nullptr;
    int32_t *labels = nullptr;

    ~TrainState() {
        if (blob) (void)hipFree(blob);
        if (loss_host) (void)hipHostFree(loss_host);
    }
};

}  // namespace

struct iefwd_instance {
    iefwd_config cfg{};
    int device = 0;
    DeviceInfo dev{};
    uint32_t head_dim = 0;

    // weights: one device allocation, carved; decode instances hold a second
    // one with the packed copies of the four matrices per layer
    void *wblob = nullptr, *pblob = nullptr;
    std::vector<LayerWeights> layers;
    float *gf = nullptr, *bef = nullptr;
    bf16_t *wh = nullptr, *bh = nullptr;

    // workspace: one device allocation, carved (sized for max_batch * max_seq)
    void *wsblob = nullptr;
    float *h = nullptr, *z = nullptr, *z2 = nullptr, *h1 = nullptr, *out = nullptr, *xstage = nullptr;
    float *stats1 = nullptr, *stats2 = nullptr;   // per-row {mean, rstd} of post-LN LayerNorms
    // KV cache (kv_cache = 1): per layer K [max_batch, H, max_seq, dh] and
    // V^T [max_batch, H, dh, max_seq rounded up to 64]
    void *kvblob = nullptr;
    std::vector<bf16_t *> kcache, vtcache;
    uint32_t kv_len = 0, kv_batch = 0;            // positions and sequences the cache holds
    float *dec_partials = nullptr;                // decode attention: per-chunk partial results
    bf16_t *hb = nullptr, *h1b = nullptr, *q = nullptr, *k = nullptr, *vt = nullptr, *ctx = nullptr,
           *u = nullptr;

    // quota
    MaskedStreams streams;
    hipStream_t stream = nullptr;
    std::vector<uint32_t> mask, pending_mask;
    bool pending = false;

    // batch state
    enum class State { Idle, InFlight, Done } state = State::Idle;
    uint32_t batch = 0, seq = 0;
    hipEvent_t ev_start = nullptr, ev_end = nullptr, ev_copy = nullptr;
    bool poisoned = false;
    bool have_batch = false;

    // per-kernel timing
    struct Timing {
        bool enabled = false;
        std::vector<std::pair<hipEvent_t, hipEvent_t>> inflight;
        double total_ms = 0;
        uint64_t launches = 0;
    } timing[IEFWD_K_COUNT];
    std::vector<hipEvent_t> event_pool;
    uint64_t kernels_launched = 0;   // every kernel this instance has launched

    std::unique_ptr<TrainState> train;   // iefwd_train_create only

    ~iefwd_instance();
};

namespace {

void check_alive(const iefwd_instance *inst) {
    if (!inst) fail(IEFWD_EINVAL, "instance is NULL");
    if (inst->poisoned) fail(IEFWD_EHIP, "instance is poisoned by an earlier HIP error; destroy it");
}

// Runs f; a HIP error inside poisons the instance.
template <class F>
void on_device(iefwd_instance *inst, F &&f) {
    try {
        hip_check(hipSetDevice(inst->device), "hipSetDevice");
        f();
    } catch (const Error &e) {
        if (e.status == IEFWD_EHIP) inst->poisoned = true;
        throw;
    }
}

hipEvent_t take_event(iefwd_instance *inst) {
    if (!inst->event_pool.empty()) {
        hipEvent_t e = inst->event_pool.back();
        inst->event_pool.pop_back();
        return e;
    }
    hipEvent_t e;
    hip_check(hipEventCreate(&e), "hipEventCreate");
    return e;
}

// Launch one kernel of class `kind`; when that class is timed the launch records
// the kernel's own start and end timestamps into a pair of events.
template <class F>
void launch(iefwd_instance *inst, uint32_t kind, const char *what, F &&f) {
    const uint64_t before = launch_count();
    auto &t = inst->timing[kind];
    if (t.enabled) {
        // the operation's first kernel records its start, its last kernel its end
        hipEvent_t e0 = take_event(inst), e1 = take_event(inst);
        armed_launch_events() = LaunchEvents{e0, e1};
        const hipError_t err = f();
        armed_launch_events() = LaunchEvents{};
        inst->kernels_launched += launch_count() - before;
        hip_check(err, what);
        t.inflight.emplace_back(e0, e1);
    } else {
        const hipError_t err = f();
        inst->kernels_launched += launch_count() - before;
        hip_check(err, what);
    }
}

void collect_timings(iefwd_instance *inst) {
    for (auto &t : inst->timing) {
        for (auto &pr : t.inflight) {
            float ms = 0;
            hip_check(hipEventElapsedTime(&ms, pr.first, pr.second), "hipEventElapsedTime");
            t.total_ms += ms;
            t.launches += 1;
            inst->event_pool.push_back(pr.first);
            inst->event_pool.push_back(pr.second);
        }
        t.inflight.clear();
    }
}

// The forward pass of one batch on inst->stream.  x: fp32 [T, d] device.
// decode_pos >= 0: one new token per sequence (I->seq == 1) at that position:
// its K and V are appended to the KV cache and it attends to positions
// 0 .. decode_pos.
void run_forward(iefwd_instance *I, const float *x, int decode_pos = -1) {
    const iefwd_config &c = I->cfg;
    const int T = (int)(I->batch * I->seq), d = (int)c.d_model, F = (int)c.d_ff;
    const int H = (int)c.n_heads, dh = (int)I->head_dim, S = (int)I->seq, B = (int)I->batch;
    const float eps = c.ln_eps;
    hipStream_t s = I->stream;
    // K and V go to the layer's KV cache when the instance keeps one (for
    // iefwd_decode), else to the per-batch buffers
    const int kv_rows = (int)c.max_seq, kv_stride = attn_seq_pad((int)c.max_seq);
    const bool decode = decode_pos >= 0;
    auto qkv_dst = [&](int l) {
        return c.kv_cache ? QkvDst{I->q, I->kcache[l], I->vtcache[l], S, decode ? decode_pos : 0, kv_rows,
                                   kv_stride, H, dh, d}
                          : QkvDst{I->q, I->k, I->vt, S, 0, S, attn_seq_pad(S), H, dh, d};
    };

    // QKV projection, attention and the output projection with its residual:
    // either a plain fp32 residual or one rebuilt from LayerNorm row statistics.
    // decode steps of up to 16 sequences use the skinny GEMM (bound by reading
    // the weights once); everything else the tiled GEMM
    // the skinny GEMM can also normalise its activations itself (a pre-LN
    // block's LayerNorm fused into the product that consumes it)
    const bool skinny = decode && T <= 16;
    const bool fuse_ln = skinny && c.pre_ln && skinny_ln_fits(T, d);
    const int n_cu = (int)mask_popcount(I->mask, I->dev.n_cu);   // the quota this batch runs on
    // j: which of the layer's four matrices (its packed copy serves decode steps)
    auto gemm = [&](Epi epi, const bf16_t *a, const LayerWeights &w, int j, const bf16_t *bias, const float *resid,
                    void *out, int N, int K, const QkvDst *qkv, const LnResid *ln_resid, const LnIn *ln_in = nullptr) {
        const bf16_t *wt = j == 0 ? w.wqkv : j == 1 ? w.wo : j == 2 ? w.w1 : w.w2;
        if (skinny && !ln_resid)
            return launch_gemm_skinny(epi, a, wt, bias, resid, out, T, N, K, qkv, s, ln_in, w.packed[j],
                                      w.packed_groups[j]);
        return launch_gemm(epi, a, wt, bias, resid, out, T, N, K, qkv, s, ln_resid, nullptr, n_cu);
    };
    auto attention_block = [&](int l, const bf16_t *y_bf16, const LayerWeights &w, const float *resid,
                               const LnResid *ln_resid, float *dst, const LnIn *ln_in = nullptr) {
        const QkvDst qd = qkv_dst(l);
        launch(I, IEFWD_K_QKV, "qkv gemm", [&] {
            return gemm(Epi::Qkv, y_bf16, w, 0, w.bqkv, nullptr, nullptr, 3 * d, d, &qd, nullptr, ln_in);
        });
        launch(I, IEFWD_K_ATTN, "attention", [&] {
            if (decode)
                return launch_decode_attention(I->q, qd.k, qd.vt, I->ctx, B, H, decode_pos + 1, dh, qd.k_rows,
                                               qd.vt_stride, I->dec_partials, s);
            return launch_attention(I->q, qd.k, qd.vt, I->ctx, B, H, S, dh, c.causal != 0, s, qd.k_rows,
                                    qd.vt_stride);
        });
        launch(I, IEFWD_K_OUTPROJ, "out-proj gemm", [&] {
            return gemm(ln_resid ? Epi::BiasLnResidF32 : Epi::BiasResidF32, I->ctx, w, 1, w.bo, resid, dst, d, d,
                        nullptr, ln_resid);
        });
    };
    auto ffn_block = [&](const bf16_t *y_bf16, const LayerWeights &w, const float *resid, const LnResid *ln_resid,
                         float *dst, const LnIn *ln_in = nullptr) {
        launch(I, IEFWD_K_FFN1, "ffn1 gemm", [&] {
            return gemm(Epi::BiasGeluBf16, y_bf16, w, 2, w.b1, nullptr, I->u, F, d, nullptr, nullptr, ln_in);
        });
        launch(I, IEFWD_K_FFN2, "ffn2 gemm", [&] {
            return gemm(ln_resid ? Epi::BiasLnResidF32 : Epi::BiasResidF32, I->u, w, 3, w.b2, resid, dst, d, F,
                        nullptr, ln_resid);
        });
    };
    auto ln = [&](const float *src, const float *g, const float *b, float *o32, bf16_t *o16, float *stats) {
        launch(I, IEFWD_K_LN, "layernorm",
               [&] { return launch_layernorm(src, g, b, o32, o16, T, d, eps, s, stats); });
    };
    auto ln_head = [&](const float *src, const float *g, const float *b) {
        launch(I, IEFWD_K_LN, "ln+head", [&] {
            return launch_ln_head(src, g, b, I->wh, I->bh, I->out, T, d, (int)c.n_out, eps, s);
        });
    };

    const int L = (int)c.n_layers;
    if (!c.pre_ln) {
        // post-LN: X1 = LN1(X + Attn(X)); X' = LN2(X1 + FFN(X1)).  The LayerNorms
        // write only the bf16 GEMM operand and {mean, rstd}; the fp32 residual
        // LN(z) is rebuilt in the epilogue of the GEMM that adds to it.
        launch(I, IEFWD_K_LN, "cast", [&] { return launch_cast_bf16(x, I->hb, (size_t)T * d, s); });
        for (int l = 0; l < L; ++l) {
            const LayerWeights &w = I->layers[l];
            if (l == 0) {
                attention_block(l, I->hb, w, x, nullptr, I->z);
            } else {
                const LayerWeights &prev = I->layers[l - 1];
                const LnResid r2{I->z2, I->stats2, prev.g2, prev.be2};
                attention_block(l, I->hb, w, nullptr, &r2, I->z);
            }
            ln(I->z, w.g1, w.be1, nullptr, I->h1b, I->stats1);
            const LnResid r1{I->z, I->stats1, w.g1, w.be1};
            ffn_block(I->h1b, w, nullptr, &r1, I->z2);
            if (l + 1 < L)
                ln(I->z2, w.g2, w.be2, nullptr, I->hb, I->stats2);
            else if (c.n_out > 0)
                ln_head(I->z2, w.g2, w.be2);
            else
                ln(I->z2, w.g2, w.be2, I->out, nullptr, nullptr);
        }
    } else {
        // pre-LN: X1 = X + Attn(LN1(X)); X' = X1 + FFN(LN2(X1)); final LN
        const float *xcur = x;
        for (int l = 0; l < L; ++l) {
            const LayerWeights &w = I->layers[l];
            if (fuse_ln) {
                const LnIn ln1{xcur, w.g1, w.be1, eps}, ln2{I->h1, w.g2, w.be2, eps};
                attention_block(l, nullptr, w, xcur, nullptr, I->h1, &ln1);
                ffn_block(nullptr, w, I->h1, nullptr, I->h, &ln2);
            } else {
                ln(xcur, w.g1, w.be1, nullptr, I->hb, nullptr);
                attention_block(l, I->hb, w, xcur, nullptr, I->h1);
                ln(I->h1, w.g2, w.be2, nullptr, I->hb, nullptr);
                ffn_block(I->hb, w, I->h1, nullptr, I->h);
            }
            xcur = I->h;
        }
        if (c.n_out > 0)
            ln_head(xcur, I->gf, I->bef);
        else
            ln(xcur, I->gf, I->bef, I->out, nullptr, nullptr);
    }
}

size_t out_width(const iefwd_config &c) { return c.n_out > 0 ? c.n_out : c.d_model; }

void upload_weights(iefwd_instance *I) {
    const iefwd_config &c = I->cfg;
    const uint32_t d = c.d_model, F = c.d_ff, L = c.n_layers;
    // sizes (elements)
    const size_t per_layer_bf16 = (size_t)3 * d * d + 3 * d + (size_t)d * d + d + (size_t)d * F + F + (size_t)F * d + d;
    const size_t per_layer_f32 = 4 * (size_t)d;
    size_t bytes = 0;
    auto reserve = [&](size_t n) { size_t off = bytes; bytes = round_up(bytes + n, 256); return off; };
    std::vector<size_t> offs;
    for (uint32_t l = 0; l < L; ++l) {
        offs.push_back(reserve((size_t)3 * d * d * 2));
        offs.push_back(reserve((size_t)3 * d * 2));
        offs.push_back(reserve((size_t)d * d * 2));
        offs.push_back(reserve((size_t)d * 2));
        offs.push_back(reserve((size_t)d * F * 2));
        offs.push_back(reserve((size_t)F * 2));
        offs.push_back(reserve((size_t)F * d * 2));
        offs.push_back(reserve((size_t)d * 2));
        for (int i = 0; i < 4; ++i) offs.push_back(reserve((size_t)d * 4));
    }
    const size_t g_off = reserve((size_t)d * 4), b_off = reserve((size_t)d * 4);
    const size_t wh_off = reserve((size_t)std::max<uint32_t>(c.n_out, 1) * d * 2);
    const size_t bh_off = reserve((size_t)std::max<uint32_t>(c.n_out, 1) * 2);
    (void)per_layer_bf16;
    (void)per_layer_f32;

    if (hipMalloc(&I->wblob, bytes) != hipSuccess) {
        (void)hipGetLastError();
        I->wblob = nullptr;
        fail(IEFWD_ENOMEM, "device allocation of weights failed");
    }
    char *base = static_cast<char *>(I->wblob);

    std::vector<uint16_t> stage16((size_t)std::max<size_t>((size_t)3 * d * d, (size_t)d * F));
    std::vector<float> stage32(d);
    const double ws = c.w_std, bs = c.b_std, ls = c.ln_std, qs = c.qk_std;
    const uint64_t seed = c.seed;
    auto put16 = [&](size_t off, size_t n) {
        hip_check(hipMemcpy(base + off, stage16.data(), n * 2, hipMemcpyHostToDevice), "weight upload");
    };
    auto put32 = [&](size_t off, size_t n) {
        hip_check(hipMemcpy(base + off, stage32.data(), n * 4, hipMemcpyHostToDevice), "weight upload");
    };

    I->layers.resize(L);
    size_t oi = 0;
    for (uint32_t l = 0; l < L; ++l) {
        LayerWeights &w = I->layers[l];
        auto at16 = [&](size_t off) { return reinterpret_cast<bf16_t *>(base + off); };
        auto at32 = [&](size_t off) { return reinterpret_cast<float *>(base + off); };
        // slot 0: Wqkv [d, 3d]; columns [0, 2d) are the Q and K blocks
        generate_matrix_transposed(tensor_key(seed, l, 0), d, 3 * d, 2 * d, ws, qs, stage16.data());
        w.wqkv = at16(offs[oi]); put16(offs[oi++], (size_t)3 * d * d);
        generate_vector_bf16(tensor_key(seed, l, 1), 3 * d, bs, stage16.data());
        w.bqkv = at16(offs[oi]); put16(offs[oi++], 3 * d);
        generate_matrix_transposed(tensor_key(seed, l, 2), d, d, 0, ws, 0.0, stage16.data());
        w.wo = at16(offs[oi]); put16(offs[oi++], (size_t)d * d);
        generate_vector_bf16(tensor_key(seed, l, 3), d, bs, stage16.data());
        w.bo = at16(offs[oi]); put16(offs[oi++], d);
        generate_matrix_transposed(tensor_key(seed, l, 6), d, F, 0, ws, 0.0, stage16.data());
        w.w1 = at16(offs[oi]); put16(offs[oi++], (size_t)d * F);
        generate_vector_bf16(tensor_key(seed, l, 7), F, bs, stage16.data());
        w.b1 = at16(offs[oi]); put16(offs[oi++], F);
        generate_matrix_transposed(tensor_key(seed, l, 8), F, d, 0, ws, 0.0, stage16.data());
        w.w2 = at16(offs[oi]); put16(offs[oi++], (size_t)F * d);
        generate_vector_bf16(tensor_key(seed, l, 9), d, bs, stage16.data());
        w.b2 = at16(offs[oi]); put16(offs[oi++], d);
        generate_vector_f32(tensor_key(seed, l, 4), d, 1.0, ls, stage32.data());
        w.g1 = at32(offs[oi]); put32(offs[oi++], d);
        generate_vector_f32(tensor_key(seed, l, 5), d, 0.0, ls, stage32.data());
        w.be1 = at32(offs[oi]); put32(offs[oi++], d);
        generate_vector_f32(tensor_key(seed, l, 10), d, 1.0, ls, stage32.data());
        w.g2 = at32(offs[oi]); put32(offs[oi++], d);
        generate_vector_f32(tensor_key(seed, l, 11), d, 0.0, ls, stage32.data());
        w.be2 = at32(offs[oi]); put32(offs[oi++], d);
    }
    generate_vector_f32(tensor_key(seed, L, 12), d, 1.0, ls, stage32.data());
    I->gf = reinterpret_cast<float *>(base + g_off); put32(g_off, d);
    generate_vector_f32(tensor_key(seed, L, 13), d, 0.0, ls, stage32.data());
    I->bef = reinterpret_cast<float *>(base + b_off); put32(b_off, d);
    I->wh = reinterpret_cast<bf16_t *>(base + wh_off);
    I->bh = reinterpret_cast<bf16_t *>(base + bh_off);
    if (c.n_out > 0) {
        generate_matrix_transposed(tensor_key(seed, L, 14), d, c.n_out, 0, ws, 0.0, stage16.data());
        put16(wh_off, (size_t)c.n_out * d);
        generate_vector_bf16(tensor_key(seed, L, 15), c.n_out, bs, stage16.data());
        put16(bh_off, c.n_out);
    }
}

// Decode instances: the packed copy of each layer's four matrices, for the
// K-group count a decode step of up to 4 sequences uses (with the pre-LN
// LayerNorm fused into the QKV and FFN-up products).  Larger decode batches of
// matrices whose group count differs read the row-major weights.
void pack_decode_weights(iefwd_instance *I) {
    const iefwd_config &c = I->cfg;
    const int d = (int)c.d_model, F = (int)c.d_ff;
    const bool ln = skinny_ln_fits(1, d);
    const int shape[4][2] = {{3 * d, d}, {d, d}, {F, d}, {d, F}};
    const bool fused[4] = {ln, false, ln, false};
    size_t bytes = 0;
    std::vector<size_t> offs;
    for (uint32_t l = 0; l < c.n_layers; ++l)
        for (int j = 0; j < 4; ++j) {
            offs.push_back(bytes);
            bytes = round_up(bytes + (size_t)shape[j][0] * shape[j][1] * 2, 256);
        }
    if (hipMalloc(&I->pblob, bytes) != hipSuccess) {
        (void)hipGetLastError();
        I->pblob = nullptr;
        fail(IEFWD_ENOMEM, "device allocation of the packed decode weights failed");
    }
    char *base = static_cast<char *>(I->pblob);
    size_t oi = 0;
    for (uint32_t l = 0; l < c.n_layers; ++l) {
        LayerWeights &w = I->layers[l];
        const bf16_t *src[4] = {w.wqkv, w.wo, w.w1, w.w2};
        for (int j = 0; j < 4; ++j) {
            const int N = shape[j][0], K = shape[j][1];
            const int g = skinny_groups(1, N, K, fused[j]);
            bf16_t *dst = reinterpret_cast<bf16_t *>(base + offs[oi++]);
            hip_check(launch_skinny_pack(src[j], dst, N, K, g, I->stream), "weight packing");
            w.packed[j] = dst;
            w.packed_groups[j] = g;
        }
    }
    hip_check(hipStreamSynchronize(I->stream), "hipStreamSynchronize");
}

void alloc_workspace(iefwd_instance *I) {
    const iefwd_config &c = I->cfg;
    const size_t T = (size_t)c.max_batch * c.max_seq, d = c.d_model, F = c.d_ff;
    const size_t spad = (size_t)attn_seq_pad((int)c.max_seq);
    size_t bytes = 0;
    auto reserve = [&](size_t n) { size_t off = bytes; bytes = round_up(bytes + n, 256); return off; };
    const size_t o_h = reserve(T * d * 4), o_z = reserve(T * d * 4), o_h1 = reserve(T * d * 4);
    const size_t o_z2 = reserve(T * d * 4), o_s1 = reserve(T * 8), o_s2 = reserve(T * 8);
    const size_t o_out = reserve(T * out_width(c) * 4), o_x = reserve(T * d * 4);
    const size_t o_hb = reserve(T * d * 2), o_h1b = reserve(T * d * 2), o_q = reserve(T * d * 2);
    const size_t o_k = reserve(T * d * 2), o_vt = reserve((size_t)c.max_batch * d * spad * 2);
    const size_t o_ctx = reserve(T * d * 2), o_u = reserve(T * F * 2);
    if (hipMalloc(&I->wsblob, bytes) != hipSuccess) {
        (void)hipGetLastError();
        I->wsblob = nullptr;
        fail(IEFWD_ENOMEM, "device allocation of the workspace failed");
    }
    char *b = static_cast<char *>(I->wsblob);
    I->h = reinterpret_cast<float *>(b + o_h);
    I->z = reinterpret_cast<float *>(b + o_z);
    I->h1 = reinterpret_cast<float *>(b + o_h1);
    I->z2 = reinterpret_cast<float *>(b + o_z2);
    I->stats1 = reinterpret_cast<float *>(b + o_s1);
    I->stats2 = reinterpret_cast<float *>(b + o_s2);
    I->out = reinterpret_cast<float *>(b + o_out);
    I->xstage = reinterpret_cast<float *>(b + o_x);
    I->hb = reinterpret_cast<bf16_t *>(b + o_hb);
    I->h1b = reinterpret_cast<bf16_t *>(b + o_h1b);
    I->q = reinterpret_cast<bf16_t *>(b + o_q);
    I->k = reinterpret_cast<bf16_t *>(b + o_k);
    I->vt = reinterpret_cast<bf16_t *>(b + o_vt);
    I->ctx = reinterpret_cast<bf16_t *>(b + o_ctx);
    I->u = reinterpret_cast<bf16_t *>(b + o_u);

    if (c.kv_cache) {
        const size_t kbytes = round_up((size_t)c.max_batch * d * c.max_seq * 2, 256);
        const size_t vbytes = round_up((size_t)c.max_batch * d * spad * 2, 256);
        const size_t bh = (size_t)c.max_batch * c.n_heads;
        const size_t pbytes = round_up(bh * kDecodeMaxChunks * (I->head_dim + 2) * 4, 256);
        if (hipMalloc(&I->kvblob, (kbytes + vbytes) * c.n_layers + pbytes) != hipSuccess) {
            (void)hipGetLastError();
            I->kvblob = nullptr;
            fail(IEFWD_ENOMEM, "device allocation of the KV cache failed");
        }
        char *kv = static_cast<char *>(I->kvblob);
        for (uint32_t l = 0; l < c.n_layers; ++l) {
            I->kcache.push_back(reinterpret_cast<bf16_t *>(kv + l * (kbytes + vbytes)));
            I->vtcache.push_back(reinterpret_cast<bf16_t *>(kv + l * (kbytes + vbytes) + kbytes));
        }
        I->dec_partials = reinterpret_cast<float *>(kv + c.n_layers * (kbytes + vbytes));
    }
}

void apply_pending_quota(iefwd_instance *I) {
    if (!I->pending) return;
    hipStream_t next = nullptr;
    hip_check(I->streams.acquire(I->pending_mask, &next), "hipExtStreamCreateWithCUMask");
    if (next != I->stream) {
        // order the new queue after everything the old one was given
        if (I->have_batch) hip_check(hipStreamWaitEvent(next, I->ev_end, 0), "hipStreamWaitEvent");
        I->stream = next;
        I->mask = I->pending_mask;
    }
    I->pending = false;
}

void wait_batch(iefwd_instance *I) {
    if (I->state != iefwd_instance::State::InFlight) return;
    hip_check(hipEventSynchronize(I->ev_end), "hipEventSynchronize");
    collect_timings(I);
    I->state = iefwd_instance::State::Done;
}

// ----------------------------------------------------------------------------- training

void validate_train(const iefwd_config &c, const iefwd_train_params &p) {
    if (p.abi_version != IEFWD_ABI_VERSION) fail(IEFWD_EVERSION, "train params abi_version mismatch");
    auto bad = [](const char *m) { fail(IEFWD_EINVAL, m); };
    if (c.pre_ln) bad("training covers post-LN stacks (pre_ln = 0)");
    if (c.kv_cache) bad("a training instance keeps no KV cache");
    if (c.n_out < 1) bad("training needs a head: n_out classes in [1, 16]");
    if (c.d_model / c.n_heads != 64) bad("training needs head dim 64");
    if (c.max_seq > 128) bad("training needs max_seq <= 128");
    if (!(p.lr >= 0.f) || !std::isfinite(p.lr)) bad("lr must be finite and >= 0");
    if (!(p.beta1 >= 0.f && p.beta1 < 1.f) || !(p.beta2 >= 0.f && p.beta2 < 1.f)) bad("betas must be in [0, 1)");
    if (!(p.eps > 0.f) || !std::isfinite(p.eps)) bad("eps must be positive and finite");
    if (!(p.weight_decay >= 0.f) || !std::isfinite(p.weight_decay)) bad("weight_decay must be finite and >= 0");
}

// Allocates the training state and initialises the fp32 master weights from
// the instance's stored bf16 / fp32 weights, the moments to zero and W^T.
// Rows of each column-sum partials region for T tokens: the most any first
// stage writes (bias gradients: T / 64; LayerNorm parameters:
// ln_backward_partials; the head: colsum_partials).
int colpart_rows(int T, int d) {
    return std::max({T / 64, ln_backward_partials(T, d), colsum_partials(T)});
}

void train_alloc(iefwd_instance *I, const iefwd_train_params &hp) {
    const iefwd_config &c = I->cfg;
    auto ts = std::make_unique<TrainState>();
    TrainState &t = *ts;
    t.hp = hp;
    const size_t L = c.n_layers, d = c.d_model, F = c.d_ff, T = (size_t)c.max_batch * c.max_seq;
    const size_t no = c.n_out, spad = (size_t)attn_seq_pad((int)c.max_seq);

    // parameter segments, each padded to the AdamW block
    const size_t blk = (size_t)adamw_block();
    const size_t counts[12] = {3 * d * d, 3 * d, d * d, d, d, d, F * d, F, d * F, d, d, d};
    size_t n = 0;
    t.off.resize(L);
    for (size_t l = 0; l < L; ++l)
        for (int k = 0; k < 12; ++k) {
            t.off[l][k] = n;
            n += round_up(counts[k], blk);
        }
    t.off_wh = n;
    n += round_up(no * d, blk);
    t.off_bh = n;
    n += round_up(no, blk);
    t.n_params = n;

    // one allocation
    size_t bytes = 0;
    auto reserve = [&](size_t b) { size_t o = bytes; bytes = round_up(bytes + b, 256); return o; };
    const size_t o_master = reserve(n * 4), o_grad = reserve(n * 4), o_m = reserve(n * 4), o_v = reserve(n * 4);
    const size_t n_seg = 12 * L + 2;
    const size_t o_segs = reserve(n_seg * sizeof(AdamSegment)), o_blk = reserve(n / blk * 4);
    std::vector<std::array<size_t, 4>> o_wt(L);
    for (size_t l = 0; l < L; ++l)
        o_wt[l] = {reserve(3 * d * d * 2), reserve(d * d * 2), reserve(d * F * 2), reserve(F * d * 2)};
    struct SavedOff { size_t hb, q, k, vt, ctx, h1b, v, u, z1, st1, z2, st2; };
    std::vector<SavedOff> o_sv(L);
    for (size_t l = 0; l < L; ++l)
        o_sv[l] = {reserve(T * d * 2), reserve(T * d * 2), reserve(T * d * 2), reserve(c.max_batch * d * spad * 2),
                   reserve(T * d * 2), reserve(T * d * 2), reserve(T * F * 2), reserve(T * F * 2),
                   reserve(T * d * 4), reserve(T * 8), reserve(T * d * 4), reserve(T * 8)};
    const size_t wide = std::max(F, 3 * d);
    const size_t o_dxa = reserve(T * d * 4), o_dxb = reserve(T * d * 4), o_dz = reserve(T * d * 4);
    const size_t o_xl = reserve(T * d * 4), o_loss = reserve(T * 4), o_dl = reserve(T * no * 4);
    // partial column sums of every bias / LayerNorm gradient of one layer (or of the head), each at most
    // [colpart_rows, n]
    const size_t o_colpart = reserve((size_t)colpart_rows((int)T, (int)d) * std::max(9 * d + F, no * d + no + 1) * 4);
    const size_t o_lsum = reserve(4);
    const size_t o_dzb = reserve(T * d * 2), o_dvb = reserve(T * F * 2), o_dctx = reserve(T * d * 2);
    const size_t o_dqkv = reserve(T * 3 * d * 2), o_ta = reserve(wide * T * 2), o_tb = reserve(wide * T * 2);
    const size_t o_zero = reserve(wide * 2), o_lab = reserve(T * 4);
    const size_t o_ascr = reserve(attention_backward_scratch((int)c.max_batch, (int)c.n_heads) * 2);
    if (hipMalloc(&t.blob, bytes) != hipSuccess) {
        (void)hipGetLastError();
        t.blob = nullptr;
        fail(IEFWD_ENOMEM, "device allocation of the training state failed");
    }
    if (hipHostMalloc(reinterpret_cast<void **>(&t.loss_host), 4) != hipSuccess) {
        (void)hipGetLastError();
        t.loss_host = nullptr;
        fail(IEFWD_ENOMEM, "pinned host allocation failed");
    }
    char *b = static_cast<char *>(t.blob);
    auto f32 = [&](size_t o) { return reinterpret_cast<float *>(b + o); };
    auto b16 = [&](size_t o) { return reinterpret_cast<bf16_t *>(b + o); };
    t.master = f32(o_master);
    t.grad = f32(o_grad);
    t.mom1 = f32(o_m);
    t.mom2 = f32(o_v);
    t.segs_d = reinterpret_cast<AdamSegment *>(b + o_segs);
    t.blk_seg_d = reinterpret_cast<uint32_t *>(b + o_blk);
    for (size_t l = 0; l < L; ++l) {
        t.wt.push_back({b16(o_wt[l][0]), b16(o_wt[l][1]), b16(o_wt[l][2]), b16(o_wt[l][3])});
        const SavedOff &o = o_sv[l];
        t.saved.push_back({b16(o.hb), b16(o.q), b16(o.k), b16(o.vt), b16(o.ctx), b16(o.h1b), b16(o.v), b16(o.u),
                           f32(o.z1), f32(o.st1), f32(o.z2), f32(o.st2)});
    }
    t.dxa = f32(o_dxa); t.dxb = f32(o_dxb); t.dz = f32(o_dz); t.xl = f32(o_xl); t.loss_t = f32(o_loss);
    t.dlogits = f32(o_dl); t.colpart = f32(o_colpart); t.loss_sum = f32(o_lsum);
    t.dzb = b16(o_dzb); t.dvb = b16(o_dvb); t.dctx = b16(o_dctx); t.dqkv = b16(o_dqkv); t.ta = b16(o_ta);
    t.tb = b16(o_tb); t.zero_bias = b16(o_zero); t.attn_scratch = b16(o_ascr);
    t.labels = reinterpret_cast<int32_t *>(b + o_lab);

    // segments: where each tensor's updated value goes (the forward's copy)
    for (size_t l = 0; l < L; ++l) {
        const LayerWeights &w = I->layers[l];
        void *outs[12] = {w.wqkv, w.bqkv, w.wo, w.bo, w.g1, w.be1, w.w1, w.b1, w.w2, w.b2, w.g2, w.be2};
        for (int k = 0; k < 12; ++k) {
            const bool is_f32 = k == 4 || k == 5 || k == 10 || k == 11;
            const bool decay = k == 0 || k == 2 || k == 6 || k == 8;
            t.segs.push_back({t.off[l][k], counts[k], outs[k], is_f32 ? 0 : 1, decay ? 1 : 0});
        }
    }
    t.segs.push_back({t.off_wh, no * d, I->wh, 1, 1});
    t.segs.push_back({t.off_bh, no, I->bh, 1, 0});
    std::vector<uint32_t> blk_seg(n / blk);
    for (size_t si = 0; si < t.segs.size(); ++si) {
        const size_t b0 = t.segs[si].offset / blk, b1 = (t.segs[si].offset + t.segs[si].count + blk - 1) / blk;
        for (size_t bb = b0; bb < b1; ++bb) blk_seg[bb] = (uint32_t)si;
    }
    t.n_blocks = (int)blk_seg.size();
    hipStream_t s = I->stream;
    hip_check(hipMemcpyAsync(t.segs_d, t.segs.data(), t.segs.size() * sizeof(AdamSegment), hipMemcpyHostToDevice, s),
              "segment upload");
    hip_check(hipMemcpyAsync(t.blk_seg_d, blk_seg.data(), blk_seg.size() * 4, hipMemcpyHostToDevice, s),
              "segment upload");
    hip_check(hipMemsetAsync(t.master, 0, n * 4, s), "hipMemsetAsync");
    hip_check(hipMemsetAsync(t.grad, 0, n * 4, s), "hipMemsetAsync");
    hip_check(hipMemsetAsync(t.mom1, 0, n * 4, s), "hipMemsetAsync");
    hip_check(hipMemsetAsync(t.mom2, 0, n * 4, s), "hipMemsetAsync");
    hip_check(hipMemsetAsync(t.zero_bias, 0, wide * 2, s), "hipMemsetAsync");
    for (const AdamSegment &sg : t.segs) {
        if (sg.out_bf16)
            hip_check(launch_bf16_to_f32(static_cast<const bf16_t *>(sg.out), t.master + sg.offset, sg.count, s),
                      "master init");
        else
            hip_check(hipMemcpyAsync(t.master + sg.offset, sg.out, sg.count * 4, hipMemcpyDeviceToDevice, s),
                      "master init");
    }
    for (size_t l = 0; l < L; ++l) {
        const LayerWeights &w = I->layers[l];
        hip_check(launch_transpose_bf16(w.wqkv, t.wt[l].wqkv, (int)(3 * d), (int)d, s), "transpose");
        hip_check(launch_transpose_bf16(w.wo, t.wt[l].wo, (int)d, (int)d, s), "transpose");
        hip_check(launch_transpose_bf16(w.w1, t.wt[l].w1, (int)F, (int)d, s), "transpose");
        hip_check(launch_transpose_bf16(w.w2, t.wt[l].w2, (int)d, (int)F, s), "transpose");
    }
    hip_check(hipStreamSynchronize(s), "hipStreamSynchronize");
    I->train = std::move(ts);
}

// One training step on I->stream: forward with saved activations, loss, backward,
// AdamW, then W^T refreshed.  x fp32 [B*S, d] and labels int32 [B*S] on the device.
void train_run(iefwd_instance *I, const float *x) {
    TrainState &t = *I->train;
    const iefwd_config &c = I->cfg;
    const int B = (int)I->batch, S = (int)I->seq, T = B * S, d = (int)c.d_model, F = (int)c.d_ff;
    const int H = (int)c.n_heads, dh = (int)I->head_dim, L = (int)c.n_layers, no = (int)c.n_out;
    const int spad = attn_seq_pad(S);
    const float eps = c.ln_eps;
    const bool causal = c.causal != 0;
    hipStream_t s = I->stream;
    const int n_cu = (int)mask_popcount(I->mask, I->dev.n_cu);   // the quota this step runs on
    auto fwd = [&](uint32_t kind, const char *what, auto &&f) { launch(I, kind, what, f); };
    auto bwd_gemm = [&](const char *what, auto &&f) { launch(I, IEFWD_K_BWD_GEMM, what, f); };
    auto bwd = [&](const char *what, auto &&f) { launch(I, IEFWD_K_BWD, what, f); };
    // Column sums of [T, n] matrices into dst [n], two fixed-order stages: the
    // partials of row blocks when the source is ready (into t.colpart at column
    // offset `col`, colpart_rows(T, d) rows per region), the last stages of a
    // layer's sums together in one launch.  Bias gradients take their partials
    // from the transpose of the output gradient (64-row blocks), LayerNorm
    // parameters from the LayerNorm backward (16-row blocks for d <= 1024), the
    // head's sums from 256-row chunks.
    const int parts = colsum_partials(T), blocks64 = T / 64, ln_parts = ln_backward_partials(T, d);
    std::vector<ColsumJob> finals;
    auto region = [&](int col) { return t.colpart + (size_t)colpart_rows(T, d) * col; };
    auto colsum = [&](const void *src, bool is_bf16, int n, float *dst, int col) {
        bwd("column sums", [&] { return launch_colsum(src, is_bf16, region(col), T, n, 256, s); });
        finals.push_back({region(col), dst, parts, n});
    };
    auto flush_finals = [&] {
        bwd("column sums", [&] { return launch_colsums(finals.data(), (int)finals.size(), s); });
        finals.clear();
    };
    auto transposes = [&](std::initializer_list<TransposeJob> jobs) {
        bwd("transpose", [&] { return launch_transposes(jobs.begin(), (int)jobs.size(), s); });
    };

    // ---- forward, saving what the backward needs
    for (int l = 0; l < L; ++l) {
        const LayerWeights &w = I->layers[l];
        const TrainState::Saved &sv = t.saved[l];
        if (l == 0)
            fwd(IEFWD_K_LN, "cast", [&] { return launch_cast_bf16(x, sv.hb, (size_t)T * d, s); });
        const QkvDst qd{sv.q, sv.k, sv.vt, S, 0, S, spad, H, dh, d};
        fwd(IEFWD_K_QKV, "qkv gemm",
            [&] {
                return launch_gemm(Epi::Qkv, sv.hb, w.wqkv, w.bqkv, nullptr, nullptr, T, 3 * d, d, &qd, s, nullptr,
                                   nullptr, n_cu);
            });
        fwd(IEFWD_K_ATTN, "attention",
            [&] { return launch_attention(sv.q, sv.k, sv.vt, sv.ctx, B, H, S, dh, causal, s, S, spad); });
        if (l == 0) {
            fwd(IEFWD_K_OUTPROJ, "out-proj gemm", [&] {
                return launch_gemm(Epi::BiasResidF32, sv.ctx, w.wo, w.bo, x, sv.z1, T, d, d, nullptr, s,
                                   nullptr, nullptr, n_cu);
            });
        } else {
            const LayerWeights &pw = I->layers[l - 1];
            const LnResid r{t.saved[l - 1].z2, t.saved[l - 1].st2, pw.g2, pw.be2};
            fwd(IEFWD_K_OUTPROJ, "out-proj gemm", [&] {
                return launch_gemm(Epi::BiasLnResidF32, sv.ctx, w.wo, w.bo, nullptr, sv.z1, T, d, d, nullptr, s,
                                   &r, nullptr, n_cu);
            });
        }
        fwd(IEFWD_K_LN, "layernorm",
            [&] { return launch_layernorm(sv.z1, w.g1, w.be1, nullptr, sv.h1b, T, d, eps, s, sv.st1); });
        fwd(IEFWD_K_FFN1, "ffn1 gemm",
            [&] { return launch_gemm(Epi::BiasBf16, sv.h1b, w.w1, w.b1, nullptr, sv.v, T, F, d, nullptr, s,
                                     nullptr, nullptr, n_cu); });
        fwd(IEFWD_K_FFN1, "gelu", [&] { return launch_gelu(sv.v, sv.u, (size_t)T * F, s); });
        const LnResid r1{sv.z1, sv.st1, w.g1, w.be1};
        fwd(IEFWD_K_FFN2, "ffn2 gemm", [&] {
            return launch_gemm(Epi::BiasLnResidF32, sv.u, w.w2, w.b2, nullptr, sv.z2, T, d, F, nullptr, s,
                               &r1, nullptr, n_cu);
        });
        if (l + 1 < L)
            fwd(IEFWD_K_LN, "layernorm", [&] {
                return launch_layernorm(sv.z2, w.g2, w.be2, nullptr, t.saved[l + 1].hb, T, d, eps, s, sv.st2);
            });
    }
    // last LayerNorm + head + cross-entropy; dX of the last layer's output into dxa
    {
        const LayerWeights &w = I->layers[L - 1];
        const TrainState::Saved &sv = t.saved[L - 1];
        fwd(IEFWD_K_LN, "head + loss", [&] {
            return launch_head_loss(sv.z2, w.g2, w.be2, I->wh, I->bh, t.labels, t.xl, sv.st2, I->out, t.loss_t,
                                    t.dlogits, t.dxa, T, d, no, eps, 1.0f / (float)T, s);
        });
        bwd("head partials", [&] { return launch_head_partials(t.dlogits, t.xl, region(0), T, d, no, s); });
        finals.push_back({region(0), t.grad + t.off_wh, parts, no * d});
        colsum(t.dlogits, false, no, t.grad + t.off_bh, no * d);
        colsum(t.loss_t, false, 1, t.loss_sum, no * d + no);
        flush_finals();
    }

    // ---- backward, last layer first; dxa holds dL/d(layer output)
    // LayerNorm backward (dz fp32 and bf16) with its parameters' partial sums
    auto ln_backward = [&](const float *dy, const float *z, const float *st, const float *gamma, size_t off_g,
                           size_t off_b, int col) {
        bwd("layernorm backward", [&] {
            return launch_ln_backward_params(dy, z, st, gamma, t.dz, t.dzb, region(col), region(col + d), T, d, s);
        });
        finals.push_back({region(col), t.grad + off_g, ln_parts, d});
        finals.push_back({region(col + d), t.grad + off_b, ln_parts, d});
    };
    // column offsets of a layer's partial sums in t.colpart
    const int c_ln2 = 0, c_b2 = 2 * d, c_b1 = 3 * d, c_ln1 = 3 * d + F, c_bo = 5 * d + F, c_bqkv = 6 * d + F;
    for (int l = L - 1; l >= 0; --l) {
        const LayerWeights &w = I->layers[l];
        const TrainState::Saved &sv = t.saved[l];
        const TrainState::Transposed &wt = t.wt[l];
        const auto &o = t.off[l];
        // LN2: dz2 (fp32 in dz, bf16 in dzb)
        ln_backward(t.dxa, sv.z2, sv.st2, w.g2, o[10], o[11], c_ln2);
        // FFN-down: dW2 = dz2^T u, db2, dv = (dz2 W2) GELU'(v)
        transposes({{t.dzb, t.ta, T, d, region(c_b2)}, {sv.u, t.tb, T, F}});
        finals.push_back({region(c_b2), t.grad + o[9], blocks64, d});
        bwd_gemm("dW2 gemm", [&] {
            return launch_gemm(Epi::F32, t.ta, t.tb, nullptr, nullptr, t.grad + o[8], d, F, T, nullptr, s,
                               nullptr, nullptr, n_cu);
        });
        bwd_gemm("dv gemm", [&] {
            return launch_gemm(Epi::GeluBwdBf16, t.dzb, wt.w2, nullptr, nullptr, t.dvb, T, F, d, nullptr, s, nullptr,
                               sv.v, n_cu);
        });
        // FFN-up: dW1 = dv^T X1, db1, dX1 = dz2 + dv W1
        transposes({{t.dvb, t.ta, T, F, region(c_b1)}, {sv.h1b, t.tb, T, d}});
        finals.push_back({region(c_b1), t.grad + o[7], blocks64, F});
        bwd_gemm("dW1 gemm", [&] {
            return launch_gemm(Epi::F32, t.ta, t.tb, nullptr, nullptr, t.grad + o[6], F, d, T, nullptr, s,
                               nullptr, nullptr, n_cu);
        });
        bwd_gemm("dX1 gemm", [&] {
            return launch_gemm(Epi::BiasResidF32, t.dvb, wt.w1, t.zero_bias, t.dz, t.dxb, T, d, F, nullptr, s,
                               nullptr, nullptr, n_cu);
        });
        // LN1: dz1
        ln_backward(t.dxb, sv.z1, sv.st1, w.g1, o[4], o[5], c_ln1);
        // out-projection: dWo = dz1^T ctx, dbo, dctx = dz1 Wo
        transposes({{t.dzb, t.ta, T, d, region(c_bo)}, {sv.ctx, t.tb, T, d}});
        finals.push_back({region(c_bo), t.grad + o[3], blocks64, d});
        bwd_gemm("dWo gemm", [&] {
            return launch_gemm(Epi::F32, t.ta, t.tb, nullptr, nullptr, t.grad + o[2], d, d, T, nullptr, s,
                               nullptr, nullptr, n_cu);
        });
        bwd_gemm("dctx gemm", [&] {
            return launch_gemm(Epi::BiasBf16, t.dzb, wt.wo, t.zero_bias, nullptr, t.dctx, T, d, d, nullptr, s,
                               nullptr, nullptr, n_cu);
        });
        // attention
        bwd("attention backward", [&] {
            return launch_attention_backward(sv.q, sv.k, sv.vt, sv.ctx, t.dctx, t.dqkv, t.attn_scratch, B, H, S, dh,
                                             spad, causal, s);
        });
        // QKV: dWqkv = dqkv^T X, dbqkv, dX = dz1 + dqkv Wqkv
        transposes({{t.dqkv, t.ta, T, 3 * d, region(c_bqkv)}, {sv.hb, t.tb, T, d}});
        finals.push_back({region(c_bqkv), t.grad + o[1], blocks64, 3 * d});
        bwd_gemm("dWqkv gemm", [&] {
            return launch_gemm(Epi::F32, t.ta, t.tb, nullptr, nullptr, t.grad + o[0], 3 * d, d, T, nullptr, s,
                               nullptr, nullptr, n_cu);
        });
        if (l > 0)
            bwd_gemm("dX gemm", [&] {
                return launch_gemm(Epi::BiasResidF32, t.dqkv, wt.wqkv, t.zero_bias, t.dz, t.dxa, T, d, 3 * d, nullptr,
                                   s, nullptr, nullptr, n_cu);
            });
        flush_finals();
    }

    // ---- AdamW over every parameter, then W^T for the next step's input gradients
    t.steps += 1;
    AdamStep st{};
    st.lr = t.hp.lr;
    st.beta1 = t.hp.beta1;
    st.beta2 = t.hp.beta2;
    st.eps = t.hp.eps;
    st.weight_decay = t.hp.weight_decay;
    st.c1 = (float)(1.0 / (1.0 - std::pow((double)t.hp.beta1, (double)t.steps)));
    st.c2 = (float)(1.0 / (1.0 - std::pow((double)t.hp.beta2, (double)t.steps)));
    launch(I, IEFWD_K_OPTIM, "adamw", [&] {
        return launch_adamw(t.master, t.grad, t.mom1, t.mom2, t.segs_d, t.blk_seg_d, t.n_blocks, st, s);
    });
    std::vector<TransposeJob> wjobs;
    for (int l = 0; l < L; ++l) {
        const LayerWeights &w = I->layers[l];
        const TrainState::Transposed &wt = t.wt[l];
        wjobs.push_back({w.wqkv, wt.wqkv, 3 * d, d});
        wjobs.push_back({w.wo, wt.wo, d, d});
        wjobs.push_back({w.w1, wt.w1, F, d});
        wjobs.push_back({w.w2, wt.w2, d, F});
    }
    for (size_t j = 0; j < wjobs.size(); j += kMaxTransposeJobs) {
        const int n = (int)std::min(wjobs.size() - j, (size_t)kMaxTransposeJobs);
        launch(I, IEFWD_K_OPTIM, "transpose", [&] { return launch_transposes(wjobs.data() + j, n, s); });
    }
    hip_check(hipMemcpyAsync(t.loss_host, t.loss_sum, 4, hipMemcpyDeviceToHost, s), "loss copy");
}

}  // namespace

iefwd_instance::~iefwd_instance() {
    if (stream) (void)hipStreamSynchronize(stream);
    streams.clear();
    for (auto &t : timing)
        for (auto &pr : t.inflight) {
            (void)hipEventDestroy(pr.first);
            (void)hipEventDestroy(pr.second);
        }
    for (hipEvent_t e : event_pool) (void)hipEventDestroy(e);
    for (hipEvent_t e : {ev_start, ev_end, ev_copy})
        if (e) (void)hipEventDestroy(e);
    train.reset();
    if (wsblob) (void)hipFree(wsblob);
    if (kvblob) (void)hipFree(kvblob);
    if (pblob) (void)hipFree(pblob);
    if (wblob) (void)hipFree(wblob);
}

// ========================================================================== fixed scratch

namespace {

// Device scratch of the allocation-free decode attention entry point: the
// per-chunk partial results (max, sum, unnormalised context) of one call.
// Each GPU the library runs on holds its own copy until the process ends; all
// calls on a GPU share it.  In host code `scratch` names a host-side stand-in,
// never the device memory: kernels get the address hipGetSymbolAddress returns
// for the current device.
constexpr size_t kNoallocScratchBytes = size_t(8) << 20;
static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_dev[kMaxScratchDevices];   // device address of `scratch` per device, once looked up

// Address of the current device's `scratch`, looked up on the first call on
// that device (with that device current).
void *scratch_on_current_device() {
    int dev = 0;
    hip_check(hipGetDevice(&dev), "hipGetDevice");
    if (dev < 0 || dev >= kMaxScratchDevices) fail(IEFWD_ENODEV, "device index beyond the scratch table");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
        void *ptr = nullptr;
        hip_check(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
        if (!ptr) fail(IEFWD_EHIP, "hipGetSymbolAddress(scratch) returned NULL");
        g_scratch_dev[dev] = ptr;
    }
    return g_scratch_dev[dev];
}

void check_decode_attention_args(const void *q, const void *k, const void *vt, void *ctx, uint32_t batch,
                                 uint32_t n_heads, uint32_t n_keys, uint32_t head_dim, uint32_t k_rows,
                                 uint32_t vt_stride) {
    if (!q || !k || !vt || !ctx) fail(IEFWD_EINVAL, "NULL pointer");
    if (batch == 0 || n_heads == 0 || (uint64_t)batch * n_heads > 65535) fail(IEFWD_EINVAL, "bad batch / heads");
    if (head_dim != 64 && head_dim != 128) fail(IEFWD_EINVAL, "head_dim must be 64 or 128");
    if (n_keys == 0 || n_keys > 8192 || k_rows < n_keys || vt_stride < n_keys || vt_stride % 64)
        fail(IEFWD_EINVAL, "need 1 <= n_keys <= 8192, k_rows >= n_keys, vt_stride >= n_keys and % 64 == 0");
}

}  // namespace

// =================================================================================== ABI

extern "C" {

void iefwd_config_init(iefwd_config *cfg) {
    if (!cfg) return;
    std::memset(cfg, 0, sizeof *cfg);
    cfg->abi_version = IEFWD_ABI_VERSION;
    cfg->ln_eps = 1e-5f;
    cfg->w_std = 0.02f;
}

int iefwd_device_info(int device, uint32_t *n_cu, uint32_t *n_xcd) {
    return guarded([&] {
        if (!n_cu || !n_xcd) fail(IEFWD_EINVAL, "NULL output pointer");
        const DeviceInfo d = query_device(device);
        *n_cu = d.n_cu;
        *n_xcd = d.n_xcd;
    });
}

int iefwd_build_cu_mask(uint32_t n_cu, uint32_t n_xcd, uint32_t quota, uint32_t first, uint32_t *mask,
                        uint32_t n_words) {
    return guarded([&] {
        if (!build_cu_mask(n_cu, n_xcd, quota, first, mask, n_words))
            fail(IEFWD_EINVAL, "invalid mask request (quota 1..n_cu, n_xcd dividing n_cu, enough words)");
    });
}

namespace {

int create_instance(const iefwd_config *cfg, const iefwd_train_params *tp, int device, iefwd_instance **out) {
    if (out) *out = nullptr;
    iefwd_instance *inst = nullptr;
    const int st = guarded([&] {
        if (!cfg || !out) fail(IEFWD_EINVAL, "NULL argument");
        validate_config(*cfg);
        if (tp) validate_train(*cfg, *tp);
        const DeviceInfo dev = query_device(device);
        hip_check(hipSetDevice(device), "hipSetDevice");
        inst = new iefwd_instance();
        inst->cfg = *cfg;
        inst->device = device;
        inst->dev = dev;
        inst->head_dim = cfg->d_model / cfg->n_heads;
        upload_weights(inst);
        alloc_workspace(inst);
        hip_check(hipEventCreate(&inst->ev_start), "hipEventCreate");
        hip_check(hipEventCreate(&inst->ev_end), "hipEventCreate");
        hip_check(hipEventCreateWithFlags(&inst->ev_copy, hipEventDisableTiming), "hipEventCreate");
        std::vector<uint32_t> all(mask_words(dev.n_cu));
        if (!build_cu_mask(dev.n_cu, dev.n_xcd, dev.n_cu, 0, all.data(), (uint32_t)all.size()))
            fail(IEFWD_ENODEV, "device CU count is not a multiple of its XCD count");
        hip_check(inst->streams.acquire(all, &inst->stream), "hipExtStreamCreateWithCUMask");
        inst->mask = all;
        if (cfg->kv_cache) pack_decode_weights(inst);
        if (tp) train_alloc(inst, *tp);
    });
    if (st != IEFWD_OK) {
        delete inst;
        return st;
    }
    *out = inst;
    return IEFWD_OK;
}

}  // namespace

int iefwd_create(const iefwd_config *cfg, int device, iefwd_instance **out) {
    return create_instance(cfg, nullptr, device, out);
}

void iefwd_train_params_init(iefwd_train_params *tp) {
    if (!tp) return;
    std::memset(tp, 0, sizeof *tp);
    tp->abi_version = IEFWD_ABI_VERSION;
    tp->lr = 1e-4f;
    tp->beta1 = 0.9f;
    tp->beta2 = 0.999f;
    tp->eps = 1e-8f;
    tp->weight_decay = 0.01f;
}

int iefwd_train_create(const iefwd_config *cfg, const iefwd_train_params *tp, int device, iefwd_instance **out) {
    if (!tp) {
        if (out) *out = nullptr;
        return guarded([&] { fail(IEFWD_EINVAL, "train params are NULL"); });
    }
    return create_instance(cfg, tp, device, out);
}

int iefwd_train_step(iefwd_instance *inst, const float *x, const int32_t *labels, uint32_t batch, uint32_t seq,
                     int inputs_are_device) {
    return guarded([&] {
        check_alive(inst);
        if (!inst->train) fail(IEFWD_ESTATE, "not a training instance (iefwd_train_create)");
        if (!x || !labels) fail(IEFWD_EINVAL, "x or labels is NULL");
        if (batch < 1 || batch > inst->cfg.max_batch) fail(IEFWD_EINVAL, "batch out of range [1, max_batch]");
        if (seq < 1 || seq > inst->cfg.max_seq) fail(IEFWD_EINVAL, "seq out of range [1, max_seq]");
        if (((uint64_t)batch * seq) % 64) fail(IEFWD_EINVAL, "batch * seq must be a multiple of 64");
        if (inst->state == iefwd_instance::State::InFlight)
            fail(IEFWD_ESTATE, "a step is already in flight; call iefwd_wait or iefwd_train_loss first");
        on_device(inst, [&] {
            apply_pending_quota(inst);
            inst->batch = batch;
            inst->seq = seq;
            const size_t T = (size_t)batch * seq, n = T * inst->cfg.d_model;
            const float *xin = x;
            const hipMemcpyKind kind = inputs_are_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice;
            hip_check(hipMemcpyAsync(inst->train->labels, labels, T * 4, kind, inst->stream), "label copy");
            if (!inputs_are_device) {
                hip_check(hipMemcpyAsync(inst->xstage, x, n * 4, hipMemcpyHostToDevice, inst->stream), "input copy");
                xin = inst->xstage;
            }
            if (!inputs_are_device) {
                hip_check(hipEventRecord(inst->ev_copy, inst->stream), "hipEventRecord");
                hip_check(hipEventSynchronize(inst->ev_copy), "hipEventSynchronize");
            }
            hip_check(hipEventRecord(inst->ev_start, inst->stream), "hipEventRecord");
            train_run(inst, xin);
            hip_check(hipEventRecord(inst->ev_end, inst->stream), "hipEventRecord");
            inst->state = iefwd_instance::State::InFlight;
            inst->have_batch = true;
        });
    });
}

int iefwd_train_loss(iefwd_instance *inst, float *loss) {
    return guarded([&] {
        check_alive(inst);
        if (!loss) fail(IEFWD_EINVAL, "loss is NULL");
        if (!inst->train) fail(IEFWD_ESTATE, "not a training instance (iefwd_train_create)");
        if (inst->train->steps == 0) fail(IEFWD_ESTATE, "no training step has run");
        on_device(inst, [&] { wait_batch(inst); });
        *loss = inst->train->loss_host[0] / (float)((uint64_t)inst->batch * inst->seq);
    });
}

int iefwd_train_steps(const iefwd_instance *inst, uint64_t *steps) {
    return guarded([&] {
        if (!inst || !steps) fail(IEFWD_EINVAL, "NULL argument");
        *steps = inst->train ? inst->train->steps : 0;
    });
}

int iefwd_train_export(iefwd_instance *inst, uint32_t layer, uint32_t slot, uint32_t what, float *host_dst,
                       size_t n_floats) {
    return guarded([&] {
        check_alive(inst);
        if (!host_dst) fail(IEFWD_EINVAL, "host_dst is NULL");
        if (!inst->train) fail(IEFWD_ESTATE, "not a training instance (iefwd_train_create)");
        if (what > IEFWD_TRAIN_MOMENT2) fail(IEFWD_EINVAL, "unknown optimiser tensor");
        const iefwd_config &c = inst->cfg;
        const TrainState &t = *inst->train;
        const size_t d = c.d_model, F = c.d_ff;
        size_t off = 0, rows = 1, cols = 0;   // logical [rows = in, cols = out]; stored [out, in]
        bool matrix = false;
        if (layer < c.n_layers) {
            if (slot > 11) fail(IEFWD_EINVAL, "per-layer slot must be 0..11");
            off = t.off[layer][slot];
            const size_t in[12] = {d, 1, d, 1, 1, 1, d, 1, F, 1, 1, 1};
            const size_t outn[12] = {3 * d, 3 * d, d, d, d, d, F, F, d, d, d, d};
            rows = in[slot];
            cols = outn[slot];
            matrix = slot == 0 || slot == 2 || slot == 6 || slot == 8;
        } else if (layer == c.n_layers && (slot == 14 || slot == 15)) {
            off = slot == 14 ? t.off_wh : t.off_bh;
            rows = slot == 14 ? d : 1;
            cols = c.n_out;
            matrix = slot == 14;
        } else {
            fail(IEFWD_EINVAL, "layer / slot out of range (the head is slots 14, 15 of layer n_layers)");
        }
        if (n_floats != rows * cols) fail(IEFWD_EINVAL, "n_floats does not match the tensor size");
        const float *base[4] = {t.master, t.grad, t.mom1, t.mom2};
        on_device(inst, [&] {
            wait_batch(inst);
            std::vector<float> stored(rows * cols);
            hip_check(hipMemcpy(stored.data(), base[what] + off, stored.size() * 4, hipMemcpyDeviceToHost),
                      "export copy");
            if (!matrix) {
                std::memcpy(host_dst, stored.data(), stored.size() * 4);
                return;
            }
            for (size_t o = 0; o < cols; ++o)
                for (size_t i = 0; i < rows; ++i) host_dst[i * cols + o] = stored[o * rows + i];
        });
    });
}

int iefwd_destroy(iefwd_instance *inst) {
    if (!inst) return IEFWD_OK;
    return guarded([&] {
        (void)hipSetDevice(inst->device);
        delete inst;
    });
}

int iefwd_set_quota_at(iefwd_instance *inst, uint32_t n_cu, uint32_t first) {
    return guarded([&] {
        check_alive(inst);
        std::vector<uint32_t> m(mask_words(inst->dev.n_cu));
        if (!build_cu_mask(inst->dev.n_cu, inst->dev.n_xcd, n_cu, first, m.data(), (uint32_t)m.size()))
            fail(IEFWD_EINVAL, "quota must be in [1, device CUs] and first below the device CUs");
        inst->pending_mask = m;
        inst->pending = true;
    });
}

int iefwd_set_quota(iefwd_instance *inst, uint32_t n_cu) { return iefwd_set_quota_at(inst, n_cu, 0); }

int iefwd_prepare_quota_at(iefwd_instance *inst, uint32_t n_cu, uint32_t first) {
    return guarded([&] {
        check_alive(inst);
        std::vector<uint32_t> m(mask_words(inst->dev.n_cu));
        if (!build_cu_mask(inst->dev.n_cu, inst->dev.n_xcd, n_cu, first, m.data(), (uint32_t)m.size()))
            fail(IEFWD_EINVAL, "quota must be in [1, device CUs] and first below the device CUs");
        hip_check(hipSetDevice(inst->device), "hipSetDevice");
        hip_check(inst->streams.prepare(m), "hipExtStreamCreateWithCUMask");
    });
}

int iefwd_set_stream_cache(iefwd_instance *inst, uint32_t capacity) {
    return guarded([&] {
        check_alive(inst);
        if (capacity < 1 || capacity > 16) fail(IEFWD_EINVAL, "capacity must be in [1, 16]");
        hip_check(hipSetDevice(inst->device), "hipSetDevice");
        hip_check(inst->streams.set_capacity(capacity), "hipStreamDestroy");
    });
}

int iefwd_set_cu_mask(iefwd_instance *inst, const uint32_t *mask, uint32_t n_words) {
    return guarded([&] {
        check_alive(inst);
        if (!mask || n_words == 0) fail(IEFWD_EINVAL, "NULL or empty mask");
        std::vector<uint32_t> m(mask_words(inst->dev.n_cu), 0u);
        for (uint32_t i = 0; i < m.size() && i < n_words; ++i) m[i] = mask[i];
        const uint32_t tail = inst->dev.n_cu % 32;
        if (tail) m.back() &= (1u << tail) - 1u;
        if (mask_popcount(m, inst->dev.n_cu) == 0) fail(IEFWD_EINVAL, "mask enables no CU of this device");
        inst->pending_mask = m;
        inst->pending = true;
    });
}

int iefwd_get_cu_mask(const iefwd_instance *inst, uint32_t *mask, uint32_t n_words) {
    return guarded([&] {
        check_alive(inst);
        if (!mask || n_words < inst->mask.size()) fail(IEFWD_EINVAL, "mask buffer too small");
        std::fill(mask, mask + n_words, 0u);
        std::copy(inst->mask.begin(), inst->mask.end(), mask);
    });
}

int iefwd_submit(iefwd_instance *inst, const float *x, uint32_t batch, uint32_t seq, int x_is_device) {
    return guarded([&] {
        check_alive(inst);
        if (!x) fail(IEFWD_EINVAL, "x is NULL");
        if (batch < 1 || batch > inst->cfg.max_batch) fail(IEFWD_EINVAL, "batch out of range [1, max_batch]");
        if (seq < 1 || seq > inst->cfg.max_seq) fail(IEFWD_EINVAL, "seq out of range [1, max_seq]");
        if (inst->state == iefwd_instance::State::InFlight)
            fail(IEFWD_ESTATE, "a batch is already in flight; call iefwd_wait or iefwd_read_logits first");
        on_device(inst, [&] {
            apply_pending_quota(inst);
            inst->batch = batch;
            inst->seq = seq;
            const size_t n = (size_t)batch * seq * inst->cfg.d_model;
            const float *xin = x;
            if (!x_is_device) {
                hip_check(hipMemcpyAsync(inst->xstage, x, n * 4, hipMemcpyHostToDevice, inst->stream), "input copy");
                hip_check(hipEventRecord(inst->ev_copy, inst->stream), "hipEventRecord");
                hip_check(hipEventSynchronize(inst->ev_copy), "hipEventSynchronize");
                xin = inst->xstage;
            }
            hip_check(hipEventRecord(inst->ev_start, inst->stream), "hipEventRecord");
            run_forward(inst, xin);
            hip_check(hipEventRecord(inst->ev_end, inst->stream), "hipEventRecord");
            inst->state = iefwd_instance::State::InFlight;
            inst->have_batch = true;
            inst->kv_len = inst->cfg.kv_cache ? seq : 0;
            inst->kv_batch = inst->cfg.kv_cache ? batch : 0;
        });
    });
}

int iefwd_decode(iefwd_instance *inst, const float *x, uint32_t batch, uint32_t pos, int x_is_device) {
    return guarded([&] {
        check_alive(inst);
        if (!x) fail(IEFWD_EINVAL, "x is NULL");
        if (!inst->cfg.kv_cache) fail(IEFWD_ESTATE, "the instance keeps no KV cache (config.kv_cache = 0)");
        if (inst->state == iefwd_instance::State::InFlight)
            fail(IEFWD_ESTATE, "a batch is already in flight; call iefwd_wait or iefwd_read_logits first");
        if (inst->kv_len == 0) fail(IEFWD_ESTATE, "no prompt in the KV cache: call iefwd_submit first");
        if (batch < 1 || batch > inst->kv_batch) fail(IEFWD_EINVAL, "batch out of range [1, sequences in the cache]");
        if (pos > inst->kv_len || pos >= inst->cfg.max_seq)
            fail(IEFWD_EINVAL, "pos must be <= the cached length and < max_seq");
        on_device(inst, [&] {
            apply_pending_quota(inst);
            inst->batch = batch;
            inst->seq = 1;
            const size_t n = (size_t)batch * inst->cfg.d_model;
            const float *xin = x;
            if (!x_is_device) {
                hip_check(hipMemcpyAsync(inst->xstage, x, n * 4, hipMemcpyHostToDevice, inst->stream), "input copy");
                hip_check(hipEventRecord(inst->ev_copy, inst->stream), "hipEventRecord");
                hip_check(hipEventSynchronize(inst->ev_copy), "hipEventSynchronize");
                xin = inst->xstage;
            }
            hip_check(hipEventRecord(inst->ev_start, inst->stream), "hipEventRecord");
            run_forward(inst, xin, (int)pos);
            hip_check(hipEventRecord(inst->ev_end, inst->stream), "hipEventRecord");
            inst->state = iefwd_instance::State::InFlight;
            inst->have_batch = true;
            inst->kv_len = pos + 1;
            inst->kv_batch = batch;
        });
    });
}

int iefwd_wait(iefwd_instance *inst) {
    return guarded([&] {
        check_alive(inst);
        on_device(inst, [&] { wait_batch(inst); });
    });
}

int iefwd_read_logits(iefwd_instance *inst, float *out, size_t n_floats, int out_is_device) {
    return guarded([&] {
        check_alive(inst);
        if (!out) fail(IEFWD_EINVAL, "out is NULL");
        if (!inst->have_batch) fail(IEFWD_ESTATE, "no batch has been submitted");
        const size_t want = (size_t)inst->batch * inst->seq * out_width(inst->cfg);
        if (n_floats != want) fail(IEFWD_EINVAL, "n_floats does not match batch * seq * output width");
        on_device(inst, [&] {
            wait_batch(inst);
            hip_check(hipMemcpyAsync(out, inst->out, want * 4,
                                     out_is_device ? hipMemcpyDeviceToDevice : hipMemcpyDeviceToHost, inst->stream),
                      "output copy");
            hip_check(hipStreamSynchronize(inst->stream), "hipStreamSynchronize");
        });
    });
}

int iefwd_last_batch_ms(iefwd_instance *inst, float *ms) {
    return guarded([&] {
        check_alive(inst);
        if (!ms) fail(IEFWD_EINVAL, "ms is NULL");
        if (inst->state != iefwd_instance::State::Done) fail(IEFWD_ESTATE, "no completed batch");
        on_device(inst, [&] { hip_check(hipEventElapsedTime(ms, inst->ev_start, inst->ev_end), "hipEventElapsedTime"); });
    });
}

int iefwd_kernels_launched(const iefwd_instance *inst, uint64_t *count) {
    return guarded([&] {
        check_alive(inst);
        if (!count) fail(IEFWD_EINVAL, "count is NULL");
        *count = inst->kernels_launched;
    });
}

int iefwd_get_stream(iefwd_instance *inst, void **hip_stream) {
    return guarded([&] {
        check_alive(inst);
        if (!hip_stream) fail(IEFWD_EINVAL, "NULL output pointer");
        *hip_stream = (void *)inst->stream;
    });
}

int iefwd_time_kernel(iefwd_instance *inst, uint32_t kind, int enable) {
    return guarded([&] {
        check_alive(inst);
        if (kind >= IEFWD_K_COUNT) fail(IEFWD_EINVAL, "unknown kernel class");
        if (inst->state == iefwd_instance::State::InFlight) fail(IEFWD_ESTATE, "a batch is in flight");
        auto &t = inst->timing[kind];
        t.enabled = enable != 0;
        t.total_ms = 0;
        t.launches = 0;
    });
}

int iefwd_kernel_time(iefwd_instance *inst, uint32_t kind, double *total_ms, uint64_t *launches) {
    return guarded([&] {
        check_alive(inst);
        if (kind >= IEFWD_K_COUNT) fail(IEFWD_EINVAL, "unknown kernel class");
        if (!total_ms || !launches) fail(IEFWD_EINVAL, "NULL output pointer");
        *total_ms = inst->timing[kind].total_ms;
        *launches = inst->timing[kind].launches;
    });
}

int iefwd_export_tensor(const iefwd_instance *cinst, uint32_t layer, uint32_t slot, void *host_dst, size_t bytes) {
    iefwd_instance *inst = const_cast<iefwd_instance *>(cinst);
    return guarded([&] {
        check_alive(inst);
        if (!host_dst) fail(IEFWD_EINVAL, "host_dst is NULL");
        const iefwd_config &c = inst->cfg;
        const size_t d = c.d_model, F = c.d_ff;
        const void *src = nullptr;
        size_t rows = 1, cols = 0, esize = 2;   // logical [rows=in, cols=out]
        bool matrix = false;
        if (layer < c.n_layers) {
            const LayerWeights &w = inst->layers[layer];
            switch (slot) {
            case 0: src = w.wqkv; rows = d; cols = 3 * d; matrix = true; break;
            case 1: src = w.bqkv; cols = 3 * d; break;
            case 2: src = w.wo; rows = d; cols = d; matrix = true; break;
            case 3: src = w.bo; cols = d; break;
            case 4: src = w.g1; cols = d; esize = 4; break;
            case 5: src = w.be1; cols = d; esize = 4; break;
            case 6: src = w.w1; rows = d; cols = F; matrix = true; break;
            case 7: src = w.b1; cols = F; break;
            case 8: src = w.w2; rows = F; cols = d; matrix = true; break;
            case 9: src = w.b2; cols = d; break;
            case 10: src = w.g2; cols = d; esize = 4; break;
            case 11: src = w.be2; cols = d; esize = 4; break;
            default: fail(IEFWD_EINVAL, "per-layer slot must be 0..11");
            }
        } else if (layer == c.n_layers) {
            switch (slot) {
            case 12: src = inst->gf; cols = d; esize = 4; break;
            case 13: src = inst->bef; cols = d; esize = 4; break;
            case 14: if (!c.n_out) fail(IEFWD_EINVAL, "no head"); src = inst->wh; rows = d; cols = c.n_out; matrix = true; break;
            case 15: if (!c.n_out) fail(IEFWD_EINVAL, "no head"); src = inst->bh; cols = c.n_out; break;
            default: fail(IEFWD_EINVAL, "global slot must be 12..15");
            }
        } else {
            fail(IEFWD_EINVAL, "layer out of range");
        }
        const size_t n = rows * cols;
        if (bytes != n * esize) fail(IEFWD_EINVAL, "bytes does not match the tensor size");
        on_device(inst, [&] {
            if (!matrix) {
                hip_check(hipMemcpy(host_dst, src, bytes, hipMemcpyDeviceToHost), "export copy");
                return;
            }
            std::vector<uint16_t> stored(n);   // device layout [cols=out, rows=in]
            hip_check(hipMemcpy(stored.data(), src, n * 2, hipMemcpyDeviceToHost), "export copy");
            uint16_t *dst = static_cast<uint16_t *>(host_dst);
            for (size_t o = 0; o < cols; ++o)
                for (size_t i = 0; i < rows; ++i) dst[i * cols + o] = stored[o * rows + i];
        });
    });
}

const char *iefwd_last_error(void) { return t_last_error.c_str(); }

// ------------------------------------------------------------------ quota controller

int iefwd_ctl_params_init(iefwd_ctl_params *p) {
    return guarded([&] {
        if (!p) fail(IEFWD_EINVAL, "params is NULL");
        const QuotaController::Params d{};
        *p = iefwd_ctl_params{};
        p->abi_version = IEFWD_ABI_VERSION;
        p->max_tokens = d.max_tokens;
        p->window = d.window;
        p->granule = d.granule;
        p->min_quota = d.min_quota;
        p->eta_violation = d.eta_violation;
        p->eta_increase = d.eta_increase;
    });
}

int iefwd_ctl_create(const iefwd_ctl_params *p, iefwd_ctl **out) {
    return guarded([&] {
        if (!out) fail(IEFWD_EINVAL, "out is NULL");
        *out = nullptr;
        if (!p) fail(IEFWD_EINVAL, "params is NULL");
        if (p->abi_version != IEFWD_ABI_VERSION) fail(IEFWD_EVERSION, "params.abi_version mismatch");
        if (p->max_tokens == 0 || p->window == 0 || p->granule == 0 || p->min_quota == 0 ||
            p->min_quota > p->max_tokens || (p->flags & ~IEFWD_CTL_TEMPORARY_YIELD) != 0)
            fail(IEFWD_EINVAL, "controller sizes out of range");
        if (!(p->eta_violation >= 0) || !(p->eta_increase >= 1) || !std::isfinite(p->eta_violation) ||
            !std::isfinite(p->eta_increase))
            fail(IEFWD_EINVAL, "eta_violation must be >= 0 and eta_increase >= 1");
        QuotaController::Params q;
        q.max_tokens = p->max_tokens;
        q.window = p->window;
        q.granule = p->granule;
        q.min_quota = p->min_quota;
        q.eta_violation = p->eta_violation;
        q.eta_increase = p->eta_increase;
        q.temporary_yield = (p->flags & IEFWD_CTL_TEMPORARY_YIELD) != 0;
        *out = reinterpret_cast<iefwd_ctl *>(new QuotaController(q));
    });
}

int iefwd_ctl_destroy(iefwd_ctl *ctl) {
    return guarded([&] { delete reinterpret_cast<QuotaController *>(ctl); });
}

int iefwd_ctl_add(iefwd_ctl *ctl, double request, double limit, int slo_sensitive, uint32_t *id) {
    return guarded([&] {
        if (!ctl || !id) fail(IEFWD_EINVAL, "NULL argument");
        if (!(request > 0) || !(limit >= request) || !(limit <= 1))
            fail(IEFWD_EINVAL, "need 0 < request <= limit <= 1");
        *id = reinterpret_cast<QuotaController *>(ctl)->add(request, limit, slo_sensitive != 0);
    });
}

int iefwd_ctl_report(iefwd_ctl *ctl, uint32_t id, uint64_t kernels, double klc_ms) {
    return guarded([&] {
        auto *c = reinterpret_cast<QuotaController *>(ctl);
        if (!c) fail(IEFWD_EINVAL, "controller is NULL");
        if (id >= c->size()) fail(IEFWD_EINVAL, "no such instance id");
        if (!std::isfinite(klc_ms)) fail(IEFWD_EINVAL, "klc_ms is not finite");
        c->report(id, kernels, klc_ms);
    });
}

int iefwd_ctl_issue(iefwd_ctl *ctl, double *tokens, uint32_t *quotas, uint32_t *firsts, uint32_t n) {
    return guarded([&] {
        auto *c = reinterpret_cast<QuotaController *>(ctl);
        if (!c) fail(IEFWD_EINVAL, "controller is NULL");
        if (n != c->size()) fail(IEFWD_EINVAL, "n must equal the number of instances");
        std::vector<double> t;
        std::vector<uint32_t> q, f;
        c->issue(t, q, f);
        for (uint32_t i = 0; i < n; ++i) {
            if (tokens) tokens[i] = t[i];
            if (quotas) quotas[i] = q[i];
            if (firsts) firsts[i] = f[i];
        }
    });
}

int iefwd_ctl_state(const iefwd_ctl *ctl, int32_t *state) {
    return guarded([&] {
        if (!ctl || !state) fail(IEFWD_EINVAL, "NULL argument");
        *state = reinterpret_cast<const QuotaController *>(ctl)->state();
    });
}

const char *iefwd_status_string(int status) {
    switch (status) {
    case IEFWD_OK: return "IEFWD_OK";
    case IEFWD_EINVAL: return "IEFWD_EINVAL";
    case IEFWD_ENODEV: return "IEFWD_ENODEV";
    case IEFWD_ENOMEM: return "IEFWD_ENOMEM";
    case IEFWD_EHIP: return "IEFWD_EHIP";
    case IEFWD_ESTATE: return "IEFWD_ESTATE";
    case IEFWD_EVERSION: return "IEFWD_EVERSION";
    default: return "IEFWD_UNKNOWN";
    }
}

// ---------------------------------------------------------------- per-kernel entry points

int iefwd_test_gemm(uint32_t epilogue, const void *a, const void *w, const void *bias, const float *resid,
                    void *out, uint32_t M, uint32_t N, uint32_t K, void *stream) {
    return guarded([&] {
        if (epilogue > IEFWD_EPI_BIAS_RESID_F32) fail(IEFWD_EINVAL, "unknown epilogue");
        if (!a || !w || !bias || !out) fail(IEFWD_EINVAL, "NULL pointer");
        if (epilogue == IEFWD_EPI_BIAS_RESID_F32 && !resid) fail(IEFWD_EINVAL, "resid is NULL");
        if (N == 0 || N % 64 || K == 0 || K % 64) fail(IEFWD_EINVAL, "N and K must be positive multiples of 64");
        if ((uint64_t)M * K >= (1ull << 31) || (uint64_t)N * K >= (1ull << 31)) fail(IEFWD_EINVAL, "too large");
        hip_check(launch_gemm((Epi)epilogue, (const bf16_t *)a, (const bf16_t *)w, (const bf16_t *)bias, resid,
                              out, (int)M, (int)N, (int)K, nullptr, (hipStream_t)stream),
                  "gemm launch");
    });
}

int iefwd_test_gemm_plan(uint32_t M, uint32_t N, uint32_t K, uint32_t align, uint32_t n_cu, uint32_t ln_residual,
                         uint32_t *k_order,
                         uint32_t *tile_order, uint32_t *tile_m, uint32_t *tile_n) {
    return guarded([&] {
        if (!k_order || !tile_order || !tile_m || !tile_n) fail(IEFWD_EINVAL, "NULL pointer");
        if (M == 0 || M > (1u << 24) || N == 0 || N % 64 || N > 65536 || K == 0 || K % 64 || K > 65536)
            fail(IEFWD_EINVAL, "need 1 <= M <= 2^24 and N, K multiples of 64 in [64, 65536]");
        if (align == 0 || align % 64 || N % align) fail(IEFWD_EINVAL, "align must be a multiple of 64 dividing N");
        if (n_cu == 0 || n_cu > 1024) fail(IEFWD_EINVAL, "n_cu must be in [1, 1024]");
        const GemmPlan p = gemm_plan((int)M, (int)N, (int)K, (int)align, (int)n_cu, ln_residual != 0);
        *k_order = p.split_order ? 1u : 0u;
        *tile_order = p.tile_split ? 1u : 0u;
        *tile_m = (uint32_t)p.bm;
        *tile_n = (uint32_t)p.bn;
    });
}

int iefwd_test_gemm_skinny(uint32_t epilogue, const void *a, const void *w, const void *bias, const float *resid,
                           void *out, uint32_t M, uint32_t N, uint32_t K, const float *ln_z, const float *ln_gamma,
                           const float *ln_beta, float ln_eps, void *stream) {
    return guarded([&] {
        if (epilogue > IEFWD_EPI_BIAS_RESID_F32) fail(IEFWD_EINVAL, "unknown epilogue");
        if (!w || !bias || !out) fail(IEFWD_EINVAL, "NULL pointer");
        if (epilogue == IEFWD_EPI_BIAS_RESID_F32 && !resid) fail(IEFWD_EINVAL, "resid is NULL");
        if (M == 0 || M > 16) fail(IEFWD_EINVAL, "M must be in [1, 16]");
        if (N == 0 || N % 16 || K == 0 || K % 32) fail(IEFWD_EINVAL, "N must be a positive multiple of 16, K of 32");
        if ((uint64_t)N * K >= (1ull << 31)) fail(IEFWD_EINVAL, "too large");
        LnIn lnin{ln_z, ln_gamma, ln_beta, ln_eps};
        if (ln_z) {
            if (!ln_gamma || !ln_beta) fail(IEFWD_EINVAL, "NULL LayerNorm parameters");
            if (!skinny_ln_fits((int)M, (int)K)) fail(IEFWD_EINVAL, "the LayerNorm prologue needs K <= 4096 and M * K <= 16384");
        } else if (!a) {
            fail(IEFWD_EINVAL, "a is NULL");
        }
        hip_check(launch_gemm_skinny((Epi)epilogue, (const bf16_t *)a, (const bf16_t *)w, (const bf16_t *)bias, resid,
                                     out, (int)M, (int)N, (int)K, nullptr, (hipStream_t)stream,
                                     ln_z ? &lnin : nullptr),
                  "skinny gemm launch");
    });
}

int iefwd_test_skinny_pack(const void *w, void *dst, uint32_t N, uint32_t K, uint32_t groups, void *stream) {
    return guarded([&] {
        if (!w || !dst) fail(IEFWD_EINVAL, "NULL pointer");
        if (groups != 1 && groups != 2 && groups != 4) fail(IEFWD_EINVAL, "groups must be 1, 2 or 4");
        if (N == 0 || N % (16 / groups) || K == 0 || K % (32 * groups))
            fail(IEFWD_EINVAL, "N must be a positive multiple of 16 / groups, K of 32 * groups");
        if ((uint64_t)N * K >= (1ull << 31)) fail(IEFWD_EINVAL, "too large");
        hip_check(launch_skinny_pack((const bf16_t *)w, (bf16_t *)dst, (int)N, (int)K, (int)groups, (hipStream_t)stream),
                  "skinny pack launch");
    });
}

int iefwd_test_gemm_skinny_packed(uint32_t epilogue, const void *a, const void *w_packed, uint32_t groups,
                                  const void *bias, const float *resid, void *out, uint32_t M, uint32_t N, uint32_t K,
                                  const float *ln_z, const float *ln_gamma, const float *ln_beta, float ln_eps,
                                  void *stream) {
    return guarded([&] {
        if (epilogue > IEFWD_EPI_BIAS_RESID_F32) fail(IEFWD_EINVAL, "unknown epilogue");
        if (!w_packed || !bias || !out) fail(IEFWD_EINVAL, "NULL pointer");
        if (epilogue == IEFWD_EPI_BIAS_RESID_F32 && !resid) fail(IEFWD_EINVAL, "resid is NULL");
        if (M == 0 || M > 16) fail(IEFWD_EINVAL, "M must be in [1, 16]");
        if (N == 0 || N % 16 || K == 0 || K % 32) fail(IEFWD_EINVAL, "N must be a positive multiple of 16, K of 32");
        if ((uint64_t)N * K >= (1ull << 31)) fail(IEFWD_EINVAL, "too large");
        LnIn lnin{ln_z, ln_gamma, ln_beta, ln_eps};
        if (ln_z) {
            if (!ln_gamma || !ln_beta) fail(IEFWD_EINVAL, "NULL LayerNorm parameters");
            if (!skinny_ln_fits((int)M, (int)K)) fail(IEFWD_EINVAL, "the LayerNorm prologue needs K <= 4096 and M * K <= 16384");
        } else if (!a) {
            fail(IEFWD_EINVAL, "a is NULL");
        }
        if ((int)groups != skinny_groups((int)M, (int)N, (int)K, ln_z != nullptr))
            fail(IEFWD_EINVAL, "the product uses another K-group count for this M, N, K");
        hip_check(launch_gemm_skinny((Epi)epilogue, (const bf16_t *)a, (const bf16_t *)w_packed, (const bf16_t *)bias,
                                     resid, out, (int)M, (int)N, (int)K, nullptr, (hipStream_t)stream,
                                     ln_z ? &lnin : nullptr, (const bf16_t *)w_packed, (int)groups),
                  "skinny gemm launch");
    });
}

int iefwd_test_skinny_groups(uint32_t M, uint32_t N, uint32_t K, int ln, uint32_t *groups) {
    return guarded([&] {
        if (!groups) fail(IEFWD_EINVAL, "groups is NULL");
        if (M == 0 || M > 16 || N == 0 || N % 16 || K == 0 || K % 32) fail(IEFWD_EINVAL, "bad shape");
        *groups = (uint32_t)skinny_groups((int)M, (int)N, (int)K, ln != 0);
    });
}

int iefwd_test_gemm_qkv(const void *a, const void *w, const void *bias, void *q, void *k, void *vt,
                        uint32_t batch, uint32_t seq, uint32_t d_model, uint32_t n_heads, void *stream) {
    return guarded([&] {
        if (!a || !w || !bias || !q || !k || !vt) fail(IEFWD_EINVAL, "NULL pointer");
        if (d_model == 0 || d_model % 64 || n_heads == 0 || d_model % n_heads) fail(IEFWD_EINVAL, "bad d_model / n_heads");
        const uint32_t dh = d_model / n_heads;
        if (dh % 8) fail(IEFWD_EINVAL, "head dim must be a multiple of 8");
        if (batch == 0 || seq == 0) fail(IEFWD_EINVAL, "empty batch");
        const uint64_t M = (uint64_t)batch * seq;
        if (M * d_model >= (1ull << 31)) fail(IEFWD_EINVAL, "too large");
        QkvDst qd{(bf16_t *)q, (bf16_t *)k, (bf16_t *)vt, (int)seq, 0, (int)seq, attn_seq_pad((int)seq),
                  (int)n_heads, (int)dh, (int)d_model};
        hip_check(launch_gemm(Epi::Qkv, (const bf16_t *)a, (const bf16_t *)w, (const bf16_t *)bias, nullptr, nullptr,
                              (int)M, (int)(3 * d_model), (int)d_model, &qd, (hipStream_t)stream),
                  "qkv gemm launch");
    });
}

int iefwd_test_attention(const void *q, const void *k, const void *vt, void *ctx, uint32_t batch, uint32_t n_heads,
                         uint32_t seq, uint32_t head_dim, int causal, void *stream) {
    return guarded([&] {
        if (!q || !k || !vt || !ctx) fail(IEFWD_EINVAL, "NULL pointer");
        if (head_dim != 64 && head_dim != 128) fail(IEFWD_EINVAL, "head_dim must be 64 or 128");
        if (batch == 0 || n_heads == 0 || seq == 0) fail(IEFWD_EINVAL, "empty shape");
        if ((uint64_t)batch * n_heads > 65535) fail(IEFWD_EINVAL, "batch * n_heads must be <= 65535");
        hip_check(launch_attention((const bf16_t *)q, (const bf16_t *)k, (const bf16_t *)vt, (bf16_t *)ctx, (int)batch,
                                   (int)n_heads, (int)seq, (int)head_dim, causal != 0, (hipStream_t)stream),
                  "attention launch");
    });
}

int iefwd_test_layernorm(const float *z, const float *gamma, const float *beta, float *out_f32, void *out_bf16,
                         uint32_t rows, uint32_t d, float eps, void *stream) {
    return guarded([&] {
        if (!z || !gamma || !beta || (!out_f32 && !out_bf16)) fail(IEFWD_EINVAL, "NULL pointer");
        if (d < 128 || d > 4096 || d % 128) fail(IEFWD_EINVAL, "d must be a multiple of 128 in [128, 4096]");
        hip_check(launch_layernorm(z, gamma, beta, out_f32, (bf16_t *)out_bf16, (int)rows, (int)d, eps,
                                   (hipStream_t)stream),
                  "layernorm launch");
    });
}

int iefwd_test_ln_head(const float *z, const float *gamma, const float *beta, const void *wh, const void *bh,
                       float *logits, uint32_t rows, uint32_t d, uint32_t n_out, float eps, void *stream) {
    return guarded([&] {
        if (!z || !gamma || !beta || !wh || !bh || !logits) fail(IEFWD_EINVAL, "NULL pointer");
        if (d < 128 || d > 4096 || d % 128) fail(IEFWD_EINVAL, "d must be a multiple of 128 in [128, 4096]");
        if (n_out < 1 || n_out > 16) fail(IEFWD_EINVAL, "n_out must be in [1, 16]");
        hip_check(launch_ln_head(z, gamma, beta, (const bf16_t *)wh, (const bf16_t *)bh, logits, (int)rows, (int)d,
                                 (int)n_out, eps, (hipStream_t)stream),
                  "ln_head launch");
    });
}

int iefwd_test_decode_attention(const void *q, const void *k, const void *vt, void *ctx, uint32_t batch,
                                uint32_t n_heads, uint32_t n_keys, uint32_t head_dim, uint32_t k_rows,
                                uint32_t vt_stride, void *stream) {
    return guarded([&] {
        check_decode_attention_args(q, k, vt, ctx, batch, n_heads, n_keys, head_dim, k_rows, vt_stride);
        // scratch for this call only: allocated, released after the stream drains
        const size_t bh = (size_t)batch * n_heads;
        const size_t pbytes = round_up(bh * kDecodeMaxChunks * (head_dim + 2) * 4, 256);
        void *scratch = nullptr;
        hip_check(hipMalloc(&scratch, pbytes), "hipMalloc");
        struct Release {
            void *p;
            ~Release() { (void)hipFree(p); }
        } release{scratch};
        hip_check(launch_decode_attention((const bf16_t *)q, (const bf16_t *)k, (const bf16_t *)vt, (bf16_t *)ctx,
                                          (int)batch, (int)n_heads, (int)n_keys, (int)head_dim, (int)k_rows,
                                          (int)vt_stride, static_cast<float *>(scratch), (hipStream_t)stream),
                  "decode attention launch");
        hip_check(hipStreamSynchronize((hipStream_t)stream), "hipStreamSynchronize");
    });
}

int iefwd_decode_attention_noalloc(const void *q, const void *k, const void *vt, void *ctx, uint32_t batch,
                                   uint32_t n_heads, uint32_t n_keys, uint32_t head_dim, uint32_t k_rows,
                                   uint32_t vt_stride, void *stream) {
    return guarded([&] {
        check_decode_attention_args(q, k, vt, ctx, batch, n_heads, n_keys, head_dim, k_rows, vt_stride);
        const size_t need = (size_t)batch * n_heads * decode_attention_chunks((int)n_keys) * (head_dim + 2) * 4;
        if (need > kNoallocScratchBytes)
            fail(IEFWD_EINVAL, "batch * heads * chunks * (head_dim + 2) * 4 = " + std::to_string(need) +
                                   " bytes exceeds the fixed scratch of " + std::to_string(kNoallocScratchBytes));
        float *partials = static_cast<float *>(scratch_on_current_device());
        hip_check(launch_decode_attention((const bf16_t *)q, (const bf16_t *)k, (const bf16_t *)vt, (bf16_t *)ctx,
                                          (int)batch, (int)n_heads, (int)n_keys, (int)head_dim, (int)k_rows,
                                          (int)vt_stride, partials, (hipStream_t)stream),
                  "decode attention launch");
    });
}

int iefwd_test_cu_probe(void *stream, uint32_t n_groups, uint32_t *out) {
    return guarded([&] {
        if (!out) fail(IEFWD_EINVAL, "out is NULL");
        if (n_groups == 0 || n_groups > (1u << 20)) fail(IEFWD_EINVAL, "n_groups must be in [1, 2^20]");
        hip_check(launch_cu_probe(out, (int)n_groups, (hipStream_t)stream), "probe launch");
    });
}

}  // extern "C"
