// Backward-kernel launchers for one I/O dtype, chosen at build time by SNNLIF_IO.  With
// SNNLIF_GAIN=1 (and SNNLIF_SPK) the unit holds the backward of the layer fed by the previous
// layer's spikes through a per-feature gain.
#include "lif_host.h"
#include "lif_kernels.h"

#if !defined(SNNLIF_IO)
#error "build with -DSNNLIF_IO=<snn_io>"
#endif
#ifndef SNNLIF_GAIN
#define SNNLIF_GAIN 0
#endif

namespace snnlif {

#if !SNNLIF_GAIN

template <int IO>
snn_status backward_entry(int reset, const Plan& p, const LifK& k, int64_t T, int64_t N, const void* x,
                          const void* saved, const void* gs, void* gx, const float* v_in, const float* g_in,
                          float* g_out, hipStream_t s) {
    const float* sv = static_cast<const float*>(saved);
    const BwdSeg seg{v_in, g_in, g_out};
    auto go = [&](auto rst) {
        return backward_variant<IO>(p, [&](auto V, auto K, auto PIPE) {
            constexpr int R = decltype(rst)::value;
            constexpr int Vc = decltype(V)::value, Kc = decltype(K)::value;
            constexpr bool Pc = decltype(PIPE)::value;
            auto run = [&](auto blk, auto sync) {
                constexpr int B = decltype(blk)::value;
                constexpr bool S = decltype(sync)::value;
                return launch_blk(lif_backward_kernel<IO, R, Vc, Kc, Pc, B, S>, grid_for((N + Vc - 1) / Vc, B), B, s,
                                  k, T, N, x, sv, gs, gx, seg);
            };
            if constexpr (!Pc && Vc == 2) {
                if (p.blkb == kSyncBlock)
                    return p.syncb ? run(IntC<kSyncBlock>{}, std::true_type{})
                                   : run(IntC<kSyncBlock>{}, std::false_type{});
            }
            return run(IntC<kBlock>{}, std::false_type{});
        });
    };
    return reset == SNN_RESET_SOFT ? go(IntC<SNN_RESET_SOFT>{}) : go(IntC<SNN_RESET_HARD>{});
}

template snn_status backward_entry<SNNLIF_IO>(int, const Plan&, const LifK&, int64_t, int64_t, const void*,
                                              const void*, const void*, void*, const float*, const float*, float*,
                                              hipStream_t);

#else

#if !defined(SNNLIF_SPK)
#error "build the gain unit with -DSNNLIF_SPK=<snn_spk>"
#endif

template <int IO, int SPK>
snn_status backward_gain_entry(int reset, const Plan& p, const LifK& k, int64_t T, int64_t N, int64_t F,
                               const void* spikes_in, const float* gain, const void* saved, const void* gs,
                               void* gs_in, hipStream_t s) {
    const uint8_t* si = static_cast<const uint8_t*>(spikes_in);
    const float* sv = static_cast<const float*>(saved);
    auto go = [&](auto rst) {
        return backward_variant<IO>(p, [&](auto V, auto K, auto PIPE) {
            constexpr int R = decltype(rst)::value;
            constexpr int Vc = decltype(V)::value, Kc = decltype(K)::value;
            if constexpr (decltype(PIPE)::value) {
                return SNN_E_UNSUPPORTED;   // the gain-fed layer's plan never double-buffers
            } else {
                return launch(lif_backward_gain_kernel<IO, SPK, R, Vc, Kc>, grid_for((N + Vc - 1) / Vc), s, k,
                              T, N, F, si, gain, p.row_bytes, sv, gs, gs_in);
            }
        });
    };
    return reset == SNN_RESET_SOFT ? go(IntC<SNN_RESET_SOFT>{}) : go(IntC<SNN_RESET_HARD>{});
}

template snn_status backward_gain_entry<SNNLIF_IO, SNNLIF_SPK>(int, const Plan&, const LifK&, int64_t, int64_t,
                                                               int64_t, const void*, const float*, const void*,
                                                               const void*, void*, hipStream_t);

#endif

}  // namespace snnlif
