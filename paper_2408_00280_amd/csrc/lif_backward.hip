// Backward-kernel launcher for one I/O dtype, chosen at build time by SNNLIF_IO.
#include "lif_host.h"
#include "lif_kernels.h"

#if !defined(SNNLIF_IO)
#error "build with -DSNNLIF_IO=<snn_io>"
#endif

namespace snnlif {
namespace {

template <int IO, int RESET, int V, bool PIPE>
snn_status backward_v(const LifK& k, int64_t T, int64_t N, const void* x, const float* sv, const void* gs, void* gx,
                      hipStream_t s) {
    constexpr int K = chunk_steps(IO, V, PIPE);
    return launch(lif_backward_kernel<IO, RESET, V, K, PIPE>, grid_for((N + V - 1) / V), s, k, T, N, x, sv, gs, gx);
}

template <int IO, int RESET>
snn_status backward_plan(const Plan& p, const LifK& k, int64_t T, int64_t N, const void* x, const void* saved,
                         const void* gs, void* gx, hipStream_t s) {
    const float* sv = static_cast<const float*>(saved);
    switch (p.vb * 2 + int(p.pipe)) {
        case 8: return backward_v<IO, RESET, 4, false>(k, T, N, x, sv, gs, gx, s);
        case 9: return backward_v<IO, RESET, 4, true>(k, T, N, x, sv, gs, gx, s);
        case 4: return backward_v<IO, RESET, 2, false>(k, T, N, x, sv, gs, gx, s);
        case 5: return backward_v<IO, RESET, 2, true>(k, T, N, x, sv, gs, gx, s);
        case 2: return backward_v<IO, RESET, 1, false>(k, T, N, x, sv, gs, gx, s);
        default: return backward_v<IO, RESET, 1, true>(k, T, N, x, sv, gs, gx, s);
    }
}

}  // namespace

template <int IO>
snn_status backward_entry(int reset, const Plan& p, const LifK& k, int64_t T, int64_t N, const void* x,
                          const void* saved, const void* gs, void* gx, hipStream_t s) {
    return reset == SNN_RESET_SOFT ? backward_plan<IO, SNN_RESET_SOFT>(p, k, T, N, x, saved, gs, gx, s)
                                   : backward_plan<IO, SNN_RESET_HARD>(p, k, T, N, x, saved, gs, gx, s);
}

template snn_status backward_entry<SNNLIF_IO>(int, const Plan&, const LifK&, int64_t, int64_t, const void*,
                                              const void*, const void*, void*, hipStream_t);

}  // namespace snnlif
