// Launchers of the stack fused across depth: the forward for one (I/O dtype, spike format)
// pair (SNNLIF_IO, SNNLIF_SPK), or with SNNLIF_STACK_BWD=1 the backward for one I/O dtype.
#include "lif_host.h"
#include "lif_kernels.h"

#if !defined(SNNLIF_IO)
#error "build with -DSNNLIF_IO=<snn_io>"
#endif
#ifndef SNNLIF_STACK_BWD
#define SNNLIF_STACK_BWD 0
#endif

namespace snnlif {
namespace {

// Calls f(V, K, L) with the plan's lane width and chunk and the layer count as tags.
template <typename F>
snn_status stack_variant(const StackPlan& p, int L, F&& f) {
    auto by_k = [&](auto V, auto Lc) -> snn_status {
        switch (p.k) {
            case 4: return f(V, IntC<4>{}, Lc);
            case 8: return f(V, IntC<8>{}, Lc);
            case 16: return f(V, IntC<16>{}, Lc);
        }
        return SNN_E_UNSUPPORTED;
    };
    auto by_l = [&](auto V) -> snn_status {
        switch (L) {
            case 2: return by_k(V, IntC<2>{});
            case 3: return by_k(V, IntC<3>{});
        }
        return SNN_E_UNSUPPORTED;
    };
    switch (p.v) {
        case 2: return by_l(IntC<2>{});
        case 1: return by_l(IntC<1>{});
    }
    return SNN_E_UNSUPPORTED;
}

}  // namespace

#if !SNNLIF_STACK_BWD

#if !defined(SNNLIF_SPK)
#error "build the stack forward with -DSNNLIF_SPK=<snn_spk>"
#endif

template <int IO, int SPK>
snn_status stack_forward_entry(int reset, int L, const StackPlan& p, const LifK& k, int64_t T, int64_t N, int64_t F,
                               const void* x, const float* gains, void* spikes, void* hidden, void* saved,
                               float* v_out, hipStream_t s) {
    uint8_t* sp = static_cast<uint8_t*>(spikes);
    uint8_t* hd = static_cast<uint8_t*>(hidden);
    float* sv = static_cast<float*>(saved);
    const dim3 g = grid_for(p.lanes);
    const bool out = hidden != nullptr || v_out != nullptr;
    auto go = [&](auto rst) {
        return stack_variant(p, L, [&](auto V, auto K, auto Lc) {
            constexpr int R = decltype(rst)::value;
            constexpr int Vc = decltype(V)::value, Kc = decltype(K)::value, Lv = decltype(Lc)::value;
            return out ? launch(lif_stack_forward_kernel<IO, SPK, R, Vc, Kc, Lv, true>, g, s, k, T, N, F, x, gains, sp,
                                hd, p.row_bytes, sv, v_out)
                       : launch(lif_stack_forward_kernel<IO, SPK, R, Vc, Kc, Lv, false>, g, s, k, T, N, F, x, gains, sp,
                                hd, p.row_bytes, sv, v_out);
        });
    };
    return reset == SNN_RESET_SOFT ? go(IntC<SNN_RESET_SOFT>{}) : go(IntC<SNN_RESET_HARD>{});
}

template snn_status stack_forward_entry<SNNLIF_IO, SNNLIF_SPK>(int, int, const StackPlan&, const LifK&, int64_t,
                                                               int64_t, int64_t, const void*, const float*, void*,
                                                               void*, void*, float*, hipStream_t);

#else

template <int IO>
snn_status stack_backward_entry(int reset, int L, const StackPlan& p, const LifK& k, int64_t T, int64_t N, int64_t F,
                                const void* x, const float* gains, const void* saved, const void* gs, void* gx,
                                hipStream_t s) {
    const float* sv = static_cast<const float*>(saved);
    auto go = [&](auto rst) {
        return stack_variant(p, L, [&](auto V, auto K, auto Lc) {
            constexpr int R = decltype(rst)::value;
            constexpr int Vc = decltype(V)::value, Kc = decltype(K)::value, Lv = decltype(Lc)::value;
            return launch(lif_stack_backward_kernel<IO, R, Vc, Kc, Lv>, grid_for((N + Vc - 1) / Vc), s, k, T, N, F, x,
                          gains, sv, gs, gx);
        });
    };
    return reset == SNN_RESET_SOFT ? go(IntC<SNN_RESET_SOFT>{}) : go(IntC<SNN_RESET_HARD>{});
}

template snn_status stack_backward_entry<SNNLIF_IO>(int, int, const StackPlan&, const LifK&, int64_t, int64_t, int64_t,
                                                    const void*, const float*, const void*, const void*, void*,
                                                    hipStream_t);

#endif

}  // namespace snnlif
