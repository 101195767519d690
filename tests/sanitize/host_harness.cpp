// Host-only driver for AddressSanitizer / UndefinedBehaviorSanitizer runs, built with g++
// (no GPU code): the library's argument checks and lane/chunk planners (lif_host.h), and the
// CPU oracle (oracle/lif_oracle.c, built with gcc beside it).  Every plan the planner can
// return must map to an instantiated kernel variant, cover every neuron and size its
// checkpoint buffer without overflow; the oracle runs on ragged, empty and non-finite
// inputs.  Exit status 0 when every invariant holds (the sanitizers abort on their own
// findings).
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <limits>
#include <vector>

#include "lif_host.h"

extern "C" {
#include "lif_oracle.h"
}

using namespace snnlif;

static int failures = 0;

#define CHECK(cond)                                                                  \
    do {                                                                             \
        if (!(cond)) {                                                               \
            std::fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
            ++failures;                                                              \
        }                                                                            \
    } while (0)

static snn_lif_cfg cfg(float decay, float th, int reset, int io, int spk) {
    snn_lif_cfg c;
    c.decay = decay;
    c.v_th = th;
    c.v_reset = 0.0f;
    c.alpha = 4.0f;
    c.reset = reset;
    c.io = io;
    c.spk = spk;
    return c;
}

static void check_cfgs() {
    const float nan = std::numeric_limits<float>::quiet_NaN(), inf = std::numeric_limits<float>::infinity();
    CHECK(check_cfg(nullptr) == SNN_E_NULL);
    snn_lif_cfg c = cfg(0.5f, 1.0f, SNN_RESET_HARD, SNN_IO_F32, SNN_SPK_U8);
    CHECK(check_cfg(&c) == SNN_OK);
    for (float d : {-0.01f, 1.01f, nan, inf, -inf}) {
        snn_lif_cfg b = c;
        b.decay = d;
        CHECK(check_cfg(&b) == SNN_E_PARAM);
    }
    for (float d : {0.0f, 1.0f}) {
        snn_lif_cfg b = c;
        b.decay = d;
        CHECK(check_cfg(&b) == SNN_OK);
    }
    for (float v : {nan, inf, -inf}) {
        snn_lif_cfg b = c;
        b.v_th = v;
        CHECK(check_cfg(&b) == SNN_E_PARAM);
        b = c;
        b.v_reset = v;
        CHECK(check_cfg(&b) == SNN_E_PARAM);
    }
    for (float a : {0.0f, -1.0f, nan, inf}) {
        snn_lif_cfg b = c;
        b.alpha = a;
        CHECK(check_cfg(&b) == SNN_E_PARAM);
    }
    for (int e : {-1, 2, 1 << 30, std::numeric_limits<int>::min()}) {
        snn_lif_cfg b = c;
        b.reset = e;
        CHECK(check_cfg(&b) == SNN_E_PARAM);
        b = c;
        b.io = e;
        CHECK(check_cfg(&b) == SNN_E_PARAM);
        b = c;
        b.spk = e + 1;   // 3 and up are out of range; 0..2 are formats
        if (e + 1 < 0 || e + 1 > 2) CHECK(check_cfg(&b) == SNN_E_PARAM);
    }
}

static void check_shapes() {
    CHECK(check_shape(0, 0) == SNN_OK);
    CHECK(check_shape(-1, 1) == SNN_E_SHAPE);
    CHECK(check_shape(1, -1) == SNN_E_SHAPE);
    CHECK(check_shape(kMaxT, 1) == SNN_OK);
    CHECK(check_shape(kMaxT + 1, 1) == SNN_E_SHAPE);
    CHECK(check_shape(1, kMaxN) == SNN_OK);
    CHECK(check_shape(1, kMaxN + 1) == SNN_E_SHAPE);
    CHECK(check_shape(int64_t(1) << 13, kMaxN) == SNN_OK);          // T N = 2^44
    CHECK(check_shape((int64_t(1) << 13) + 1, kMaxN) == SNN_E_SHAPE);
    CHECK(check_shape(kMaxT, kMaxN) == SNN_E_SHAPE);
    CHECK(check_shape(std::numeric_limits<int64_t>::max(), 2) == SNN_E_SHAPE);
    CHECK(check_shape(2, std::numeric_limits<int64_t>::max()) == SNN_E_SHAPE);
}

// The instantiated variants are the ones forward_variant / backward_variant dispatch to.
struct Probe {
    template <typename V, typename K, typename P>
    snn_status operator()(V, K, P) const {
        return SNN_OK;
    }
};

static void check_plan(const snn_lif_cfg& c, int64_t T, int64_t N) {
    const Plan p = make_plan(&c, T, N);
    CHECK(p.vf == 1 || p.vf == 2 || p.vf == 4 || p.vf == 8);
    CHECK(p.vb == 1 || p.vb == 2 || p.vb == 4);
    CHECK(N % p.vb == 0 && N % p.vf == 0);             // lanes never straddle the row end
    CHECK(p.k == 4 || p.k == 8 || p.k == 16 || p.k == 32);
    CHECK(p.blkf == kBlock || p.blkf == kSyncBlock);
    CHECK(p.blkb == kBlock || p.blkb == kSyncBlock);
    if (p.blkf == kSyncBlock) CHECK(!p.pipe && T > p.k);
    if (p.blkb == kSyncBlock) CHECK(!p.pipe && T > p.k && p.vb == 2);
    CHECK(p.lanes * p.vf >= N);
    CHECK(p.row_bytes == spike_row_bytes(&c, N));
    if (c.spk == SNN_SPK_BITS) CHECK(p.lanes * p.vf >= p.row_bytes * 8);   // every spike word written
    const int64_t chunks = (T + p.k - 1) / p.k;
    CHECK(saved_bytes(p, T, N) == (chunks > 1 ? (chunks - 1) * N * 4 : 0));
    CHECK(saved_bytes(p, T, N) <= 4 * T * N);
    snn_status fs, bs;
    if (c.io == SNN_IO_F32) {
        fs = forward_variant<SNN_IO_F32>(p, Probe{});
        bs = backward_variant<SNN_IO_F32>(p, Probe{});
    } else {
        fs = forward_variant<SNN_IO_BF16>(p, Probe{});
        bs = backward_variant<SNN_IO_BF16>(p, Probe{});
    }
    if (fs != SNN_OK || bs != SNN_OK)
        std::fprintf(stderr, "no kernel variant: io %d T %lld N %lld vf %d vb %d k %d pipe %d\n", c.io,
                     (long long)T, (long long)N, p.vf, p.vb, p.k, int(p.pipe));
    CHECK(fs == SNN_OK && bs == SNN_OK);
    // the gain-fed layer: single-buffered chunks of the same length, so the same checkpoints
    const Plan gp = make_gain_plan(&c, T, N);
    CHECK(!gp.pipe && gp.k == p.k && gp.vf == p.vf && gp.vb == p.vb && gp.lanes == p.lanes);
    CHECK(saved_bytes(gp, T, N) == saved_bytes(p, T, N));
    if (c.io == SNN_IO_F32) {
        fs = forward_variant<SNN_IO_F32>(gp, Probe{});
        bs = backward_variant<SNN_IO_F32>(gp, Probe{});
    } else {
        fs = forward_variant<SNN_IO_BF16>(gp, Probe{});
        bs = backward_variant<SNN_IO_BF16>(gp, Probe{});
    }
    if (fs != SNN_OK || bs != SNN_OK)
        std::fprintf(stderr, "no gain-fed kernel variant: io %d T %lld N %lld vf %d vb %d k %d\n", c.io,
                     (long long)T, (long long)N, gp.vf, gp.vb, gp.k);
    CHECK(fs == SNN_OK && bs == SNN_OK);
    const StackPlan s = make_stack_plan(&c, T, N);
    CHECK((s.v == 1 || s.v == 2) && N % s.v == 0);
    CHECK(s.k == 4 || s.k == 8 || s.k == 16);
    CHECK(s.lanes * s.v >= N);
    for (int L = 2; L <= kMaxStackLayers; ++L) {
        const int64_t sc = (T + s.k - 1) / s.k;
        CHECK(stack_saved_bytes(s, L, T, N) == (sc > 1 ? (sc - 1) * L * N * 4 : 0));
    }
}

static void check_plans() {
    const int64_t Ns[] = {1, 2, 3, 7, 63, 64, 65, 1000, 4096, 4097, 65536, 131072, 524288, 1000000,
                          (1 << 20) + 4, 8388608, (int64_t(1) << 22) + 2, 16777216, (int64_t(1) << 24) + 8,
                          (int64_t(1) << 24) + 1, int64_t(1) << 28, kMaxN - 1, kMaxN};
    const int64_t Ts[] = {1, 2, 3, 4, 5, 8, 9, 15, 16, 17, 31, 32, 33, 40, 64, 65, 96, 128, 192, 256, 257, 1000};
    for (int io : {SNN_IO_F32, SNN_IO_BF16})
        for (int spk : {SNN_SPK_U8, SNN_SPK_BITS, SNN_SPK_IO})
            for (int reset : {SNN_RESET_HARD, SNN_RESET_SOFT})
                for (int64_t N : Ns)
                    for (int64_t T : Ts) {
                        if (check_shape(T, N) != SNN_OK) continue;
                        check_plan(cfg(0.5f, 1.0f, reset, io, spk), T, N);
                    }
}

// ---------------------------------------------------------------- the oracle

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;

static double uniform() {   // xorshift64*, for test inputs only
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return double((rng_state * 0x2545F4914F6CDD1Dull) >> 11) / double(uint64_t(1) << 53);
}

static void run_oracle(int64_t T, int64_t B, int64_t F, int soft, bool nonfinite) {
    const int64_t N = B * F, TN = T * N;
    lif_oracle_params p = {0.75f, 1.0f, 0.125f, 4.0f, soft};
    // exact-size heap buffers, so any access past an end is reported
    std::vector<float> x(TN), v(TN), xs(3 * TN), vs(3 * TN), xn(TN), gains(2 * F);
    std::vector<uint8_t> y(TN), ys(3 * TN);
    std::vector<double> gy(TN), gx(TN), ge(TN), gr(TN), sg(3 * TN), se(3 * TN), sr(3 * TN), gn(N);
    for (int64_t i = 0; i < TN; ++i) {
        x[i] = float(2.0 * uniform() - 0.3);
        gy[i] = 2.0 * uniform() - 1.0;
    }
    if (nonfinite && TN >= 3) {
        x[0] = std::numeric_limits<float>::quiet_NaN();
        x[TN / 2] = std::numeric_limits<float>::infinity();
        x[TN - 1] = -std::numeric_limits<float>::infinity();
    }
    for (int64_t f = 0; f < 2 * F; ++f) gains[f] = float(0.5 + 1.5 * uniform());
    for (int64_t n = 0; n < N; ++n) gn[n] = uniform();
    lif_oracle_forward(&p, T, N, x.data(), nullptr, nullptr, y.data(), v.data());
    lif_oracle_backward(&p, T, N, v.data(), y.data(), gy.data(), nullptr, nullptr, gn.data(), gx.data(), ge.data(),
                        gr.data());
    lif_oracle_backward(&p, T, N, v.data(), y.data(), gy.data(), ge.data(), gr.data(), nullptr, gx.data(),
                        ge.data(), nullptr);
    lif_oracle_gain_forward(T, B, F, y.data(), gains.data(), xn.data());
    lif_oracle_gain_backward(T, B, F, gx.data(), ge.data(), gr.data(), gains.data(), gy.data(), ge.data(), gr.data());
    for (int L = 1; L <= 3; ++L) {
        lif_oracle_stack_forward(&p, L, T, B, F, x.data(), gains.data(), xs.data(), ys.data(), vs.data());
        CHECK(lif_oracle_stack_backward(&p, L, T, B, F, vs.data(), ys.data(), gains.data(), gy.data(), L & 1,
                                        sg.data(), se.data(), sr.data()) == 0);
    }
    if (!nonfinite)
        for (int64_t i = 0; i < TN; ++i) CHECK(se[i] >= std::fabs(sg[i]));
}

int main() {
    check_cfgs();
    check_shapes();
    check_plans();
    const int64_t shapes[][3] = {{0, 1, 1}, {1, 0, 3}, {1, 1, 1}, {2, 3, 5}, {17, 2, 33}, {40, 3, 7}, {5, 1, 1000}};
    for (const auto& s : shapes)
        for (int soft = 0; soft < 2; ++soft)
            for (int nf = 0; nf < 2; ++nf) run_oracle(s[0], s[1], s[2], soft, nf != 0);
    if (failures) {
        std::fprintf(stderr, "%d check(s) failed\n", failures);
        return 1;
    }
    std::printf("host harness: all checks passed\n");
    return 0;
}
