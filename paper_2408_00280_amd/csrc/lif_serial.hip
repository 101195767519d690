// Launchers of the serial (per-time-step) baseline kernels.
#include "lif_host.h"
#include "lif_kernels.h"

namespace snnlif {
namespace {

bool al(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

// Four neurons per lane when every row pointer allows 4-wide accesses (rows of a [T][N]
// tensor with N % 4 != 0 only have element alignment), else one.
template <int IO, int SPK, int RESET>
snn_status serial_fwd_v(const LifK& k, int64_t N, const void* x, const float* vp, float* v, uint8_t* sp,
                        int64_t row, hipStream_t s) {
    const int64_t covered = SPK == SNN_SPK_BITS ? row * 8 : N;
    const bool vec = N % 4 == 0 && SPK != SNN_SPK_BITS && al(x, IO == SNN_IO_F32 ? 16 : 8) && al(v, 16) &&
                     (vp == nullptr || al(vp, 16)) && al(sp, SPK == SNN_SPK_U8 ? 4 : IO == SNN_IO_F32 ? 16 : 8);
    if (vec)
        return launch(lif_serial_forward_kernel<IO, SPK, RESET, 4>, grid_for(N / 4), s, k, N, x, vp, v, sp, row);
    return launch(lif_serial_forward_kernel<IO, SPK, RESET, 1>, grid_for(covered), s, k, N, x, vp, v, sp, row);
}

template <int IO, int SPK>
snn_status serial_fwd_r(int reset, const LifK& k, int64_t N, const void* x, const float* vp, float* v, uint8_t* sp,
                        int64_t row, hipStream_t s) {
    return reset == SNN_RESET_SOFT ? serial_fwd_v<IO, SPK, SNN_RESET_SOFT>(k, N, x, vp, v, sp, row, s)
                                   : serial_fwd_v<IO, SPK, SNN_RESET_HARD>(k, N, x, vp, v, sp, row, s);
}

template <int IO>
snn_status serial_fwd_s(const snn_lif_cfg* c, const LifK& k, int64_t N, const void* x, const float* vp, float* v,
                        uint8_t* sp, int64_t row, hipStream_t s) {
    switch (c->spk) {
        case SNN_SPK_U8: return serial_fwd_r<IO, SNN_SPK_U8>(c->reset, k, N, x, vp, v, sp, row, s);
        case SNN_SPK_BITS: return serial_fwd_r<IO, SNN_SPK_BITS>(c->reset, k, N, x, vp, v, sp, row, s);
        default: return serial_fwd_r<IO, SNN_SPK_IO>(c->reset, k, N, x, vp, v, sp, row, s);
    }
}

template <int IO, int RESET>
snn_status serial_bwd_v(const LifK& k, int64_t N, const float* v, const void* gs, const float* gn, void* gx,
                        float* go, hipStream_t s) {
    const uintptr_t ai = IO == SNN_IO_F32 ? 16 : 8;
    if (N % 4 == 0 && al(v, 16) && al(gs, ai) && al(gx, ai) && (gn == nullptr || al(gn, 16)) &&
        (go == nullptr || al(go, 16)))
        return launch(lif_serial_backward_kernel<IO, RESET, 4>, grid_for(N / 4), s, k, N, v, gs, gn, gx, go);
    return launch(lif_serial_backward_kernel<IO, RESET, 1>, grid_for(N), s, k, N, v, gs, gn, gx, go);
}

}  // namespace

snn_status serial_forward_entry(const snn_lif_cfg* c, const LifK& k, int64_t N, const void* x_t,
                                const float* v_prev, float* v_t, void* spikes_t, hipStream_t s) {
    uint8_t* sp = static_cast<uint8_t*>(spikes_t);
    const int64_t row = spike_row_bytes(c, N);
    return c->io == SNN_IO_F32 ? serial_fwd_s<SNN_IO_F32>(c, k, N, x_t, v_prev, v_t, sp, row, s)
                               : serial_fwd_s<SNN_IO_BF16>(c, k, N, x_t, v_prev, v_t, sp, row, s);
}

snn_status serial_backward_entry(const snn_lif_cfg* c, const LifK& k, int64_t N, const float* v_t, const void* gs_t,
                                 const float* g_next, void* gx_t, float* g_out, hipStream_t s) {
    const bool soft = c->reset == SNN_RESET_SOFT;
    if (c->io == SNN_IO_F32)
        return soft ? serial_bwd_v<SNN_IO_F32, SNN_RESET_SOFT>(k, N, v_t, gs_t, g_next, gx_t, g_out, s)
                    : serial_bwd_v<SNN_IO_F32, SNN_RESET_HARD>(k, N, v_t, gs_t, g_next, gx_t, g_out, s);
    return soft ? serial_bwd_v<SNN_IO_BF16, SNN_RESET_SOFT>(k, N, v_t, gs_t, g_next, gx_t, g_out, s)
                : serial_bwd_v<SNN_IO_BF16, SNN_RESET_HARD>(k, N, v_t, gs_t, g_next, gx_t, g_out, s);
}

}  // namespace snnlif
