// Forward-kernel launchers for one (I/O dtype, spike format) pair, chosen at build time by
// SNNLIF_IO and SNNLIF_SPK so that the variants compile as parallel translation units.
// With SNNLIF_GAIN=1 the unit holds the layer fed by the previous layer's spikes through a
// per-feature gain instead of the layer fed by a dense input current.
#include "lif_host.h"
#include "lif_kernels.h"

#if !defined(SNNLIF_IO) || !defined(SNNLIF_SPK)
#error "build with -DSNNLIF_IO=<snn_io> -DSNNLIF_SPK=<snn_spk>"
#endif
#ifndef SNNLIF_GAIN
#define SNNLIF_GAIN 0
#endif

namespace snnlif {

#if !SNNLIF_GAIN

template <int IO, int SPK>
snn_status forward_entry(int reset, const Plan& p, const LifK& k, int64_t T, int64_t N, const void* x,
                         void* spikes, void* saved, float* v_out, const float* v_in, float* v_last,
                         hipStream_t s) {
    uint8_t* sp = static_cast<uint8_t*>(spikes);
    float* sv = static_cast<float*>(saved);
    auto go = [&](auto rst) {
        return forward_variant<IO>(p, [&](auto V, auto K, auto PIPE) {
            constexpr int R = decltype(rst)::value;
            constexpr int Vc = decltype(V)::value, Kc = decltype(K)::value;
            constexpr bool Pc = decltype(PIPE)::value;
            constexpr int FB = forward_batch(IO, Vc, Kc, Pc);
            auto run = [&](auto blk) {
                constexpr int B = decltype(blk)::value;
                const dim3 g = grid_for(p.lanes, B);
                return v_out ? launch_blk(lif_forward_kernel<IO, SPK, R, Vc, FB, Kc, true, Pc, B>, g, B, s, k, T, N,
                                          x, sp, p.row_bytes, sv, v_out, v_in, v_last)
                             : launch_blk(lif_forward_kernel<IO, SPK, R, Vc, FB, Kc, false, Pc, B>, g, B, s, k, T, N,
                                          x, sp, p.row_bytes, sv, v_out, v_in, v_last);
            };
            if constexpr (!Pc && Vc >= 2) {
                if (p.blkf == kSyncBlock) return run(IntC<kSyncBlock>{});
            }
            return run(IntC<kBlock>{});
        });
    };
    return reset == SNN_RESET_SOFT ? go(IntC<SNN_RESET_SOFT>{}) : go(IntC<SNN_RESET_HARD>{});
}

template snn_status forward_entry<SNNLIF_IO, SNNLIF_SPK>(int, const Plan&, const LifK&, int64_t, int64_t,
                                                         const void*, void*, void*, float*, const float*, float*,
                                                         hipStream_t);

#else

template <int IO, int SPK>
snn_status forward_gain_entry(int reset, const Plan& p, const LifK& k, int64_t T, int64_t N, int64_t F,
                              const void* spikes_in, const float* gain, void* spikes, void* saved, float* v_out,
                              hipStream_t s) {
    const uint8_t* si = static_cast<const uint8_t*>(spikes_in);
    uint8_t* sp = static_cast<uint8_t*>(spikes);
    float* sv = static_cast<float*>(saved);
    const dim3 g = grid_for(p.lanes);
    auto go = [&](auto rst) {
        return forward_variant<IO>(p, [&](auto V, auto K, auto PIPE) {
            constexpr int R = decltype(rst)::value;
            constexpr int Vc = decltype(V)::value, Kc = decltype(K)::value;
            if constexpr (decltype(PIPE)::value) {
                return SNN_E_UNSUPPORTED;   // the gain-fed layer's plan never double-buffers
            } else {
                constexpr int FB = forward_batch(IO, Vc, Kc, false);
                return v_out ? launch(lif_forward_gain_kernel<IO, SPK, R, Vc, FB, Kc, true>, g, s, k, T, N, F, si,
                                      gain, sp, p.row_bytes, sv, v_out)
                             : launch(lif_forward_gain_kernel<IO, SPK, R, Vc, FB, Kc, false>, g, s, k, T, N, F,
                                      si, gain, sp, p.row_bytes, sv, v_out);
            }
        });
    };
    return reset == SNN_RESET_SOFT ? go(IntC<SNN_RESET_SOFT>{}) : go(IntC<SNN_RESET_HARD>{});
}

template snn_status forward_gain_entry<SNNLIF_IO, SNNLIF_SPK>(int, const Plan&, const LifK&, int64_t, int64_t,
                                                              int64_t, const void*, const float*, void*, void*,
                                                              float*, hipStream_t);

#endif

}  // namespace snnlif
