// The C ABI declared in include/snn_lif.h: argument validation, the lane/chunk plan, and
// dispatch to the kernel launchers of the other translation units.
#include "lif_host.h"

using namespace snnlif;

namespace {

snn_status forward_dispatch(const snn_lif_cfg* c, const Plan& p, const LifK& k, int64_t T, int64_t N,
                            const void* x, void* spikes, void* saved, float* v_out, const float* v_in,
                            float* v_last, hipStream_t s) {
    const int r = c->reset;
    if (c->io == SNN_IO_F32) {
        switch (c->spk) {
            case SNN_SPK_U8:
                return forward_entry<SNN_IO_F32, SNN_SPK_U8>(r, p, k, T, N, x, spikes, saved, v_out, v_in, v_last, s);
            case SNN_SPK_BITS:
                return forward_entry<SNN_IO_F32, SNN_SPK_BITS>(r, p, k, T, N, x, spikes, saved, v_out, v_in, v_last, s);
            default:
                return forward_entry<SNN_IO_F32, SNN_SPK_IO>(r, p, k, T, N, x, spikes, saved, v_out, v_in, v_last, s);
        }
    }
    switch (c->spk) {
        case SNN_SPK_U8:
            return forward_entry<SNN_IO_BF16, SNN_SPK_U8>(r, p, k, T, N, x, spikes, saved, v_out, v_in, v_last, s);
        case SNN_SPK_BITS:
            return forward_entry<SNN_IO_BF16, SNN_SPK_BITS>(r, p, k, T, N, x, spikes, saved, v_out, v_in, v_last, s);
        default:
            return forward_entry<SNN_IO_BF16, SNN_SPK_IO>(r, p, k, T, N, x, spikes, saved, v_out, v_in, v_last, s);
    }
}

snn_status check_gain_shape(int64_t T, int64_t B, int64_t F) {
    if (T < 0 || B < 0 || F < 0) return SNN_E_SHAPE;
    if (B > 0 && F > kMaxN / B) return SNN_E_SHAPE;
    return check_shape(T, B * F);
}

}  // namespace

extern "C" {

const char* snn_status_str(snn_status status) {
    switch (status) {
        case SNN_OK: return "ok";
        case SNN_E_NULL: return "a required pointer is NULL";
        case SNN_E_SHAPE: return "shape out of range";
        case SNN_E_PARAM: return "hyper-parameter or enum out of range";
        case SNN_E_ALIGN: return "data pointer not 16-byte aligned";
        case SNN_E_UNSUPPORTED: return "unsupported combination";
        case SNN_E_LAUNCH: return "kernel launch rejected by the HIP runtime";
    }
    return "unknown status";
}

snn_status snn_spike_row_bytes(const snn_lif_cfg* cfg, int64_t N, size_t* bytes) {
    snn_status st = check_cfg(cfg);
    if (st != SNN_OK) return st;
    if (bytes == nullptr) return SNN_E_NULL;
    if ((st = check_shape(0, N)) != SNN_OK) return st;
    *bytes = size_t(spike_row_bytes(cfg, N));
    return SNN_OK;
}

snn_status snn_lif_saved_bytes(const snn_lif_cfg* cfg, int64_t T, int64_t N, size_t* bytes) {
    snn_status st = check_cfg(cfg);
    if (st != SNN_OK) return st;
    if (bytes == nullptr) return SNN_E_NULL;
    if ((st = check_shape(T, N)) != SNN_OK) return st;
    *bytes = (T == 0 || N == 0) ? 0 : size_t(saved_bytes(make_plan(cfg, T, N), T, N));
    return SNN_OK;
}

snn_status snn_lif_forward_seg(const snn_lif_cfg* cfg, int64_t T, int64_t N, const void* x, const float* v_in,
                               void* spikes, void* saved, float* v_last, float* v_out, void* stream) {
    snn_status st = check_cfg(cfg);
    if (st != SNN_OK) return st;
    if ((st = check_shape(T, N)) != SNN_OK) return st;
    if (T == 0 || N == 0) return SNN_OK;
    const Plan p = make_plan(cfg, T, N);
    const bool need_saved = saved_bytes(p, T, N) > 0;
    if (x == nullptr || spikes == nullptr || (need_saved && saved == nullptr)) return SNN_E_NULL;
    if (!aligned(x) || !aligned(spikes) || (saved && !aligned(saved)) || (v_out && !aligned(v_out)) ||
        (v_in && !aligned(v_in)) || (v_last && !aligned(v_last)))
        return SNN_E_ALIGN;
    return forward_dispatch(cfg, p, kernel_consts(cfg), T, N, x, spikes, need_saved ? saved : nullptr, v_out, v_in,
                            v_last, static_cast<hipStream_t>(stream));
}

snn_status snn_lif_forward(const snn_lif_cfg* cfg, int64_t T, int64_t N, const void* x, void* spikes,
                           void* saved, float* v_out, void* stream) {
    return snn_lif_forward_seg(cfg, T, N, x, nullptr, spikes, saved, nullptr, v_out, stream);
}

snn_status snn_lif_backward_seg(const snn_lif_cfg* cfg, int64_t T, int64_t N, const void* x, const float* v_in,
                                const void* saved, const void* grad_s, const float* g_in, void* grad_x,
                                float* g_out, void* stream) {
    snn_status st = check_cfg(cfg);
    if (st != SNN_OK) return st;
    if ((st = check_shape(T, N)) != SNN_OK) return st;
    if (T == 0 || N == 0) return SNN_OK;
    const Plan p = make_plan(cfg, T, N);
    const bool need_saved = saved_bytes(p, T, N) > 0;
    if (x == nullptr || grad_s == nullptr || grad_x == nullptr || (need_saved && saved == nullptr))
        return SNN_E_NULL;
    if (!aligned(x) || !aligned(grad_s) || !aligned(grad_x) || (saved && !aligned(saved)) ||
        (v_in && !aligned(v_in)) || (g_in && !aligned(g_in)) || (g_out && !aligned(g_out)))
        return SNN_E_ALIGN;
    const LifK k = kernel_consts(cfg);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const void* sv = need_saved ? saved : nullptr;
    return cfg->io == SNN_IO_F32
               ? backward_entry<SNN_IO_F32>(cfg->reset, p, k, T, N, x, sv, grad_s, grad_x, v_in, g_in, g_out, s)
               : backward_entry<SNN_IO_BF16>(cfg->reset, p, k, T, N, x, sv, grad_s, grad_x, v_in, g_in, g_out, s);
}

snn_status snn_lif_backward(const snn_lif_cfg* cfg, int64_t T, int64_t N, const void* x, const void* saved,
                            const void* grad_s, void* grad_x, void* stream) {
    return snn_lif_backward_seg(cfg, T, N, x, nullptr, saved, grad_s, nullptr, grad_x, nullptr, stream);
}

snn_status snn_gain_spikes_forward(const snn_lif_cfg* cfg, int64_t T, int64_t B, int64_t F, const void* spikes,
                                   const float* gain, void* x_next, void* stream) {
    snn_status st = check_cfg(cfg);
    if (st != SNN_OK) return st;
    if ((st = check_gain_shape(T, B, F)) != SNN_OK) return st;
    const int64_t N = B * F;
    if (T == 0 || N == 0) return SNN_OK;
    if (spikes == nullptr || gain == nullptr || x_next == nullptr) return SNN_E_NULL;
    if (!aligned(spikes) || !aligned(gain) || !aligned(x_next)) return SNN_E_ALIGN;
    return gain_forward_entry(cfg, T, N, F, spikes, spike_row_bytes(cfg, N), gain, x_next,
                              static_cast<hipStream_t>(stream));
}

snn_status snn_gain_grad_backward(const snn_lif_cfg* cfg, int64_t T, int64_t B, int64_t F, const void* grad_x_next,
                                  const float* gain, void* grad_s, void* stream) {
    snn_status st = check_cfg(cfg);
    if (st != SNN_OK) return st;
    if ((st = check_gain_shape(T, B, F)) != SNN_OK) return st;
    const int64_t N = B * F;
    if (T == 0 || N == 0) return SNN_OK;
    if (grad_x_next == nullptr || gain == nullptr || grad_s == nullptr) return SNN_E_NULL;
    if (!aligned(grad_x_next) || !aligned(gain) || !aligned(grad_s)) return SNN_E_ALIGN;
    return gain_backward_entry(cfg, T, N, F, grad_x_next, gain, grad_s, static_cast<hipStream_t>(stream));
}

snn_status snn_lif_forward_gain(const snn_lif_cfg* cfg, int64_t T, int64_t B, int64_t F, const void* spikes_in,
                                const float* gain, void* spikes, void* saved, float* v_out, void* stream) {
    snn_status st = check_cfg(cfg);
    if (st != SNN_OK) return st;
    if ((st = check_gain_shape(T, B, F)) != SNN_OK) return st;
    const int64_t N = B * F;
    if (T == 0 || N == 0) return SNN_OK;
    const Plan p = make_gain_plan(cfg, T, N);
    const bool need_saved = saved_bytes(p, T, N) > 0;
    if (spikes_in == nullptr || gain == nullptr || spikes == nullptr || (need_saved && saved == nullptr))
        return SNN_E_NULL;
    if (!aligned(spikes_in) || !aligned(gain) || !aligned(spikes) || (saved && !aligned(saved)) ||
        (v_out && !aligned(v_out)))
        return SNN_E_ALIGN;
    const LifK k = kernel_consts(cfg);
    hipStream_t s = static_cast<hipStream_t>(stream);
    void* sv = need_saved ? saved : nullptr;
    const int r = cfg->reset;
    switch (cfg->io * 4 + cfg->spk) {
        case SNN_IO_F32 * 4 + SNN_SPK_U8:
            return forward_gain_entry<SNN_IO_F32, SNN_SPK_U8>(r, p, k, T, N, F, spikes_in, gain, spikes, sv, v_out, s);
        case SNN_IO_F32 * 4 + SNN_SPK_BITS:
            return forward_gain_entry<SNN_IO_F32, SNN_SPK_BITS>(r, p, k, T, N, F, spikes_in, gain, spikes, sv, v_out, s);
        case SNN_IO_F32 * 4 + SNN_SPK_IO:
            return forward_gain_entry<SNN_IO_F32, SNN_SPK_IO>(r, p, k, T, N, F, spikes_in, gain, spikes, sv, v_out, s);
        case SNN_IO_BF16 * 4 + SNN_SPK_U8:
            return forward_gain_entry<SNN_IO_BF16, SNN_SPK_U8>(r, p, k, T, N, F, spikes_in, gain, spikes, sv, v_out, s);
        case SNN_IO_BF16 * 4 + SNN_SPK_BITS:
            return forward_gain_entry<SNN_IO_BF16, SNN_SPK_BITS>(r, p, k, T, N, F, spikes_in, gain, spikes, sv, v_out, s);
        default:
            return forward_gain_entry<SNN_IO_BF16, SNN_SPK_IO>(r, p, k, T, N, F, spikes_in, gain, spikes, sv, v_out, s);
    }
}

snn_status snn_lif_backward_gain(const snn_lif_cfg* cfg, int64_t T, int64_t B, int64_t F, const void* spikes_in,
                                 const float* gain, const void* saved, const void* grad_s, void* grad_s_in,
                                 void* stream) {
    snn_status st = check_cfg(cfg);
    if (st != SNN_OK) return st;
    if ((st = check_gain_shape(T, B, F)) != SNN_OK) return st;
    const int64_t N = B * F;
    if (T == 0 || N == 0) return SNN_OK;
    const Plan p = make_gain_plan(cfg, T, N);
    const bool need_saved = saved_bytes(p, T, N) > 0;
    if (spikes_in == nullptr || gain == nullptr || grad_s == nullptr || grad_s_in == nullptr ||
        (need_saved && saved == nullptr))
        return SNN_E_NULL;
    if (!aligned(spikes_in) || !aligned(gain) || !aligned(grad_s) || !aligned(grad_s_in) ||
        (saved && !aligned(saved)))
        return SNN_E_ALIGN;
    const LifK k = kernel_consts(cfg);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const void* sv = need_saved ? saved : nullptr;
    const int r = cfg->reset;
    switch (cfg->io * 4 + cfg->spk) {
        case SNN_IO_F32 * 4 + SNN_SPK_U8:
            return backward_gain_entry<SNN_IO_F32, SNN_SPK_U8>(r, p, k, T, N, F, spikes_in, gain, sv, grad_s, grad_s_in, s);
        case SNN_IO_F32 * 4 + SNN_SPK_BITS:
            return backward_gain_entry<SNN_IO_F32, SNN_SPK_BITS>(r, p, k, T, N, F, spikes_in, gain, sv, grad_s, grad_s_in, s);
        case SNN_IO_F32 * 4 + SNN_SPK_IO:
            return backward_gain_entry<SNN_IO_F32, SNN_SPK_IO>(r, p, k, T, N, F, spikes_in, gain, sv, grad_s, grad_s_in, s);
        case SNN_IO_BF16 * 4 + SNN_SPK_U8:
            return backward_gain_entry<SNN_IO_BF16, SNN_SPK_U8>(r, p, k, T, N, F, spikes_in, gain, sv, grad_s, grad_s_in, s);
        case SNN_IO_BF16 * 4 + SNN_SPK_BITS:
            return backward_gain_entry<SNN_IO_BF16, SNN_SPK_BITS>(r, p, k, T, N, F, spikes_in, gain, sv, grad_s, grad_s_in, s);
        default:
            return backward_gain_entry<SNN_IO_BF16, SNN_SPK_IO>(r, p, k, T, N, F, spikes_in, gain, sv, grad_s, grad_s_in, s);
    }
}

snn_status snn_lif_stack_saved_bytes(const snn_lif_cfg* cfg, int32_t L, int64_t T, int64_t N, size_t* bytes) {
    snn_status st = check_cfg(cfg);
    if (st != SNN_OK) return st;
    if (bytes == nullptr) return SNN_E_NULL;
    if ((st = check_shape(T, N)) != SNN_OK) return st;
    if (L < 2 || L > kMaxStackLayers) return SNN_E_UNSUPPORTED;
    *bytes = (T == 0 || N == 0) ? 0 : size_t(stack_saved_bytes(make_stack_plan(cfg, T, N), L, T, N));
    return SNN_OK;
}

snn_status snn_lif_stack_forward(const snn_lif_cfg* cfg, int32_t L, int64_t T, int64_t B, int64_t F, const void* x,
                                 const float* gains, void* spikes, void* hidden_spikes, void* saved, float* v_out,
                                 void* stream) {
    snn_status st = check_cfg(cfg);
    if (st != SNN_OK) return st;
    if ((st = check_gain_shape(T, B, F)) != SNN_OK) return st;
    if (L < 2 || L > kMaxStackLayers) return SNN_E_UNSUPPORTED;
    const int64_t N = B * F;
    if (T == 0 || N == 0) return SNN_OK;
    if (T > kMaxTN / (int64_t(L) * N)) return SNN_E_SHAPE;   // v_out holds L T N values
    const StackPlan p = make_stack_plan(cfg, T, N);
    const bool need_saved = stack_saved_bytes(p, L, T, N) > 0;
    if (x == nullptr || gains == nullptr || spikes == nullptr || (need_saved && saved == nullptr)) return SNN_E_NULL;
    if (!aligned(x) || !aligned(gains) || !aligned(spikes) || (hidden_spikes && !aligned(hidden_spikes)) ||
        (saved && !aligned(saved)) || (v_out && !aligned(v_out)))
        return SNN_E_ALIGN;
    const LifK k = kernel_consts(cfg);
    hipStream_t s = static_cast<hipStream_t>(stream);
    void* sv = need_saved ? saved : nullptr;
    const int r = cfg->reset;
    switch (cfg->io * 4 + cfg->spk) {
        case SNN_IO_F32 * 4 + SNN_SPK_U8:
            return stack_forward_entry<SNN_IO_F32, SNN_SPK_U8>(r, L, p, k, T, N, F, x, gains, spikes, hidden_spikes, sv, v_out, s);
        case SNN_IO_F32 * 4 + SNN_SPK_BITS:
            return stack_forward_entry<SNN_IO_F32, SNN_SPK_BITS>(r, L, p, k, T, N, F, x, gains, spikes, hidden_spikes, sv, v_out, s);
        case SNN_IO_F32 * 4 + SNN_SPK_IO:
            return stack_forward_entry<SNN_IO_F32, SNN_SPK_IO>(r, L, p, k, T, N, F, x, gains, spikes, hidden_spikes, sv, v_out, s);
        case SNN_IO_BF16 * 4 + SNN_SPK_U8:
            return stack_forward_entry<SNN_IO_BF16, SNN_SPK_U8>(r, L, p, k, T, N, F, x, gains, spikes, hidden_spikes, sv, v_out, s);
        case SNN_IO_BF16 * 4 + SNN_SPK_BITS:
            return stack_forward_entry<SNN_IO_BF16, SNN_SPK_BITS>(r, L, p, k, T, N, F, x, gains, spikes, hidden_spikes, sv, v_out, s);
        default:
            return stack_forward_entry<SNN_IO_BF16, SNN_SPK_IO>(r, L, p, k, T, N, F, x, gains, spikes, hidden_spikes, sv, v_out, s);
    }
}

snn_status snn_lif_stack_backward(const snn_lif_cfg* cfg, int32_t L, int64_t T, int64_t B, int64_t F, const void* x,
                                  const float* gains, const void* saved, const void* grad_s, void* grad_x,
                                  void* stream) {
    snn_status st = check_cfg(cfg);
    if (st != SNN_OK) return st;
    if ((st = check_gain_shape(T, B, F)) != SNN_OK) return st;
    if (L < 2 || L > kMaxStackLayers) return SNN_E_UNSUPPORTED;
    const int64_t N = B * F;
    if (T == 0 || N == 0) return SNN_OK;
    const StackPlan p = make_stack_plan(cfg, T, N);
    const bool need_saved = stack_saved_bytes(p, L, T, N) > 0;
    if (x == nullptr || gains == nullptr || grad_s == nullptr || grad_x == nullptr || (need_saved && saved == nullptr))
        return SNN_E_NULL;
    if (!aligned(x) || !aligned(gains) || !aligned(grad_s) || !aligned(grad_x) || (saved && !aligned(saved)))
        return SNN_E_ALIGN;
    const LifK k = kernel_consts(cfg);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const void* sv = need_saved ? saved : nullptr;
    return cfg->io == SNN_IO_F32
               ? stack_backward_entry<SNN_IO_F32>(cfg->reset, L, p, k, T, N, F, x, gains, sv, grad_s, grad_x, s)
               : stack_backward_entry<SNN_IO_BF16>(cfg->reset, L, p, k, T, N, F, x, gains, sv, grad_s, grad_x, s);
}

snn_status snn_lif_serial_forward_step(const snn_lif_cfg* cfg, int64_t N, const void* x_t, const float* v_prev,
                                       float* v_t, void* spikes_t, void* stream) {
    snn_status st = check_cfg(cfg);
    if (st != SNN_OK) return st;
    if ((st = check_shape(1, N)) != SNN_OK) return st;
    if (N == 0) return SNN_OK;
    if (x_t == nullptr || v_t == nullptr || spikes_t == nullptr) return SNN_E_NULL;
    const uintptr_t e = uintptr_t(io_bytes(cfg));
    const uintptr_t es = cfg->spk == SNN_SPK_U8 ? 1 : cfg->spk == SNN_SPK_BITS ? 8 : e;
    if (!aligned_to(x_t, e) || !aligned_to(v_t, 4) || !aligned_to(spikes_t, es) || (v_prev && !aligned_to(v_prev, 4)))
        return SNN_E_ALIGN;
    return serial_forward_entry(cfg, kernel_consts(cfg), N, x_t, v_prev, v_t, spikes_t,
                                static_cast<hipStream_t>(stream));
}

snn_status snn_lif_serial_backward_step(const snn_lif_cfg* cfg, int64_t N, const float* v_t, const void* grad_s_t,
                                        const float* g_next, void* grad_x_t, float* g_out, void* stream) {
    snn_status st = check_cfg(cfg);
    if (st != SNN_OK) return st;
    if ((st = check_shape(1, N)) != SNN_OK) return st;
    if (N == 0) return SNN_OK;
    if (v_t == nullptr || grad_s_t == nullptr || grad_x_t == nullptr) return SNN_E_NULL;
    const uintptr_t e = uintptr_t(io_bytes(cfg));
    if (!aligned_to(v_t, 4) || !aligned_to(grad_s_t, e) || !aligned_to(grad_x_t, e) ||
        (g_next && !aligned_to(g_next, 4)) || (g_out && !aligned_to(g_out, 4)))
        return SNN_E_ALIGN;
    return serial_backward_entry(cfg, kernel_consts(cfg), N, v_t, grad_s_t, g_next, grad_x_t, g_out,
                                 static_cast<hipStream_t>(stream));
}

}  // extern "C"
