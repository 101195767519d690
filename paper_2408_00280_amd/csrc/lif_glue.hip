// Launchers of the per-feature gain kernels placed between stacked LIF layers.
#include "lif_host.h"
#include "lif_kernels.h"

namespace snnlif {
namespace {

// Flat launches (whole rows: one contiguous run of T*N elements, pieces that never wrap
// around the features) over kFlatPieces pieces per lane; the step between a lane's pieces
// in features is kBlock * W % F.
template <int IO>
bool flat_rows(int64_t F) { return F % flat_width<IO>() == 0; }

template <int IO>
dim3 flat_grid(int64_t T, int64_t N) {
    return grid_for((T * N / flat_width<IO>() + kFlatPieces - 1) / kFlatPieces);
}

template <int IO>
int64_t flat_step(int64_t F) { return int64_t(kBlock) * flat_width<IO>() % F; }

template <int IO, int SPK>
snn_status gain_forward_io(int64_t T, int64_t N, int64_t F, const uint8_t* sp, int64_t row, const float* gain,
                           void* x_next, hipStream_t s) {
    const bool unpadded = SPK == SNN_SPK_IO || (SPK == SNN_SPK_U8 ? row == N : row * 8 == N);
    if (flat_rows<IO>(F) && unpadded)
        return launch(gain_forward_flat_kernel<IO, SPK>, flat_grid<IO>(T, N), s, T * N / flat_width<IO>(), F,
                      flat_step<IO>(F), sp, gain, x_next);
    if (N % 4 == 0)
        return launch(gain_forward_kernel<IO, SPK, 4>, grid_for(N / 4), s, T, N, F, sp, row, gain, x_next);
    return launch(gain_forward_kernel<IO, SPK, 1>, grid_for(N), s, T, N, F, sp, row, gain, x_next);
}

template <int IO>
snn_status gain_forward_spk(int spk, int64_t T, int64_t N, int64_t F, const uint8_t* sp, int64_t row,
                            const float* gain, void* x_next, hipStream_t s) {
    switch (spk) {
        case SNN_SPK_U8: return gain_forward_io<IO, SNN_SPK_U8>(T, N, F, sp, row, gain, x_next, s);
        case SNN_SPK_BITS: return gain_forward_io<IO, SNN_SPK_BITS>(T, N, F, sp, row, gain, x_next, s);
        default: return gain_forward_io<IO, SNN_SPK_IO>(T, N, F, sp, row, gain, x_next, s);
    }
}

template <int IO>
snn_status gain_backward_io(int64_t T, int64_t N, int64_t F, const void* gxn, const float* gain, void* gs,
                            hipStream_t s) {
    if (flat_rows<IO>(F))
        return launch(gain_backward_flat_kernel<IO>, flat_grid<IO>(T, N), s, T * N / flat_width<IO>(), F,
                      flat_step<IO>(F), gxn, gain, gs);
    if (N % 4 == 0) return launch(gain_backward_kernel<IO, 4>, grid_for(N / 4), s, T, N, F, gxn, gain, gs);
    return launch(gain_backward_kernel<IO, 1>, grid_for(N), s, T, N, F, gxn, gain, gs);
}

}  // namespace

snn_status gain_forward_entry(const snn_lif_cfg* c, int64_t T, int64_t N, int64_t F, const void* spikes,
                              int64_t row_bytes, const float* gain, void* x_next, hipStream_t s) {
    const uint8_t* sp = static_cast<const uint8_t*>(spikes);
    return c->io == SNN_IO_F32 ? gain_forward_spk<SNN_IO_F32>(c->spk, T, N, F, sp, row_bytes, gain, x_next, s)
                               : gain_forward_spk<SNN_IO_BF16>(c->spk, T, N, F, sp, row_bytes, gain, x_next, s);
}

snn_status gain_backward_entry(const snn_lif_cfg* c, int64_t T, int64_t N, int64_t F, const void* gx_next,
                               const float* gain, void* gs, hipStream_t s) {
    return c->io == SNN_IO_F32 ? gain_backward_io<SNN_IO_F32>(T, N, F, gx_next, gain, gs, s)
                               : gain_backward_io<SNN_IO_BF16>(T, N, F, gx_next, gain, gs, s);
}

}  // namespace snnlif
