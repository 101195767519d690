// Forward-kernel launcher for one (I/O dtype, spike format) pair, chosen at build time by
// SNNLIF_IO and SNNLIF_SPK so that the variants compile as parallel translation units.
#include "lif_host.h"
#include "lif_kernels.h"

#if !defined(SNNLIF_IO) || !defined(SNNLIF_SPK)
#error "build with -DSNNLIF_IO=<snn_io> -DSNNLIF_SPK=<snn_spk>"
#endif

namespace snnlif {
namespace {

template <int IO, int SPK, int RESET, int V, int K, bool PIPE>
snn_status forward_v(const Plan& p, const LifK& k, int64_t T, int64_t N, const void* x, uint8_t* sp, float* sv,
                     float* v_out, hipStream_t s) {
    const dim3 g = grid_for(p.lanes);
    return v_out ? launch(lif_forward_kernel<IO, SPK, RESET, V, K, true, PIPE>, g, s, k, T, N, x, sp, p.row_bytes, sv, v_out)
                 : launch(lif_forward_kernel<IO, SPK, RESET, V, K, false, PIPE>, g, s, k, T, N, x, sp, p.row_bytes, sv, v_out);
}

// The (vf, pipe) combinations the planner produces.
template <int IO, int SPK, int RESET>
snn_status forward_plan(const Plan& p, const LifK& k, int64_t T, int64_t N, const void* x, void* spikes,
                        void* saved, float* v_out, hipStream_t s) {
    uint8_t* sp = static_cast<uint8_t*>(spikes);
    float* sv = static_cast<float*>(saved);
    constexpr int K4 = chunk_steps(IO, 4, false), K4p = chunk_steps(IO, 4, true);
    constexpr int K2 = chunk_steps(IO, 2, false), K1 = chunk_steps(IO, 1, false);
    if constexpr (IO == SNN_IO_BF16) {
        if (p.vf == 8)
            return p.pipe ? forward_v<IO, SPK, RESET, 8, K4p, true>(p, k, T, N, x, sp, sv, v_out, s)
                          : forward_v<IO, SPK, RESET, 8, K4, false>(p, k, T, N, x, sp, sv, v_out, s);
    }
    switch (p.vf * 2 + int(p.pipe)) {
        case 8: return forward_v<IO, SPK, RESET, 4, K4, false>(p, k, T, N, x, sp, sv, v_out, s);
        case 9: return forward_v<IO, SPK, RESET, 4, K4p, true>(p, k, T, N, x, sp, sv, v_out, s);
        case 4: return forward_v<IO, SPK, RESET, 2, K2, false>(p, k, T, N, x, sp, sv, v_out, s);
        case 5: return forward_v<IO, SPK, RESET, 2, K2, true>(p, k, T, N, x, sp, sv, v_out, s);
        case 2: return forward_v<IO, SPK, RESET, 1, K1, false>(p, k, T, N, x, sp, sv, v_out, s);
        default: return forward_v<IO, SPK, RESET, 1, K1, true>(p, k, T, N, x, sp, sv, v_out, s);
    }
}

}  // namespace

template <int IO, int SPK>
snn_status forward_entry(int reset, const Plan& p, const LifK& k, int64_t T, int64_t N, const void* x,
                         void* spikes, void* saved, float* v_out, hipStream_t s) {
    return reset == SNN_RESET_SOFT ? forward_plan<IO, SPK, SNN_RESET_SOFT>(p, k, T, N, x, spikes, saved, v_out, s)
                                   : forward_plan<IO, SPK, SNN_RESET_HARD>(p, k, T, N, x, spikes, saved, v_out, s);
}

template snn_status forward_entry<SNNLIF_IO, SNNLIF_SPK>(int, const Plan&, const LifK&, int64_t, int64_t,
                                                         const void*, void*, void*, float*, hipStream_t);

}  // namespace snnlif
