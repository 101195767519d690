// Host-side planning and launching for the fused LIF library: argument checks, the lane /
// chunk plan shared by forward and backward, and the per-translation-unit launchers.
#pragma once
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <tuple>
#include <type_traits>
#include <utility>

#include "lif_common.h"

namespace snnlif {

inline snn_status check_cfg(const snn_lif_cfg* c) {
    if (c == nullptr) return SNN_E_NULL;
    if (!(c->decay >= 0.0f && c->decay <= 1.0f)) return SNN_E_PARAM;  // also rejects NaN
    if (!std::isfinite(c->v_th) || !std::isfinite(c->v_reset)) return SNN_E_PARAM;
    if (!(c->alpha > 0.0f) || !std::isfinite(c->alpha)) return SNN_E_PARAM;
    if (c->reset != SNN_RESET_HARD && c->reset != SNN_RESET_SOFT) return SNN_E_PARAM;
    if (c->io != SNN_IO_F32 && c->io != SNN_IO_BF16) return SNN_E_PARAM;
    if (c->spk != SNN_SPK_U8 && c->spk != SNN_SPK_BITS && c->spk != SNN_SPK_IO) return SNN_E_PARAM;
    return SNN_OK;
}

inline snn_status check_shape(int64_t T, int64_t N) {
    if (T < 0 || N < 0 || T > kMaxT || N > kMaxN) return SNN_E_SHAPE;
    if (T > 0 && N > kMaxTN / T) return SNN_E_SHAPE;
    return SNN_OK;
}

inline bool aligned_to(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }
inline bool aligned(const void* p) { return aligned_to(p, 16); }

inline int64_t io_bytes(const snn_lif_cfg* c) { return c->io == SNN_IO_F32 ? 4 : 2; }

inline int64_t spike_row_bytes(const snn_lif_cfg* c, int64_t N) {
    return c->spk == SNN_SPK_U8 ? N : c->spk == SNN_SPK_BITS ? 8 * ((N + 63) / 64) : N * io_bytes(c);
}

// Neurons per lane in the forward (vf) and the backward (vb), steps per chunk (K, also the
// checkpoint interval, sized by the backward's register budget) and whether chunks are
// double-buffered.  The same choice drives both kernels and the checkpoint layout (which
// does not depend on the lane widths), so it depends only on (cfg, T, N).
struct Plan {
    int vf;
    int vb;
    int k;
    bool pipe;
    int blkf;        // workgroup sizes of the dense forward and backward kernels
    int blkb;
    bool syncb;      // the backward's kSyncBlock workgroups meet at a barrier after each chunk
    int64_t lanes;   // lanes in the forward grid
    int64_t row_bytes;
};

// Steps per chunk for v neurons per backward lane: the backward keeps K membranes per
// neuron in VGPRs plus K rows of x and dL/dy (twice the rows when double-buffered).  Large
// bf16 layers (not double-buffered) take 32 steps at 2 neurons per lane instead: half the
// checkpoint traffic, and bf16 rows take half the registers (make_plan).
constexpr int chunk_steps(int v) { return v == 1 ? 32 : 16; }

// A layer of T <= K steps is one chunk and keeps no checkpoint; it runs with the shortest
// of these chunk lengths that holds T, so that registers sized for K steps do not cap the
// occupancy of short-lived waves.
constexpr int kShortChunks[] = {4, 8, 16};

// Lanes that fill the chip with 16 waves per CU (256 CUs x 16 x 64).
constexpr int64_t kFillLanes = int64_t(256) * 16 * 64;

// Workgroup size for layers of several chunks that are not double-buffered.  Rows lie
// 16-32 MiB apart, each in its own 2 MiB page, and a wave uses a few hundred bytes of each;
// as waves drift apart along a long walk, the pages in use at once outgrow the per-CU
// address-translation cache.  16 waves that start together and meet at a barrier after
// every chunk share the translations of the same rows' pages.  Measured against
// 256-lane workgroups: forward -4% (bf16, T = 256) to -6.5% (fp32, T = 128 and 256);
// fp32 backward -1.5% / -5% / -6.5% / -2.5% at T = 32 / 64 / 128 / 256 (N = 8.4M).  The
// bf16 backward (32-step chunks, one such workgroup per CU) with the barrier is 1.3-2.6%
// faster than without it at T = 64 / 96 / 128 / 192 in every run (21 runs, five boxes),
// but at T = 256 it ran 13% slower in about half the runs, so it takes the barrier only
// for layers of at most kSyncBf16Chunks chunks; without one it is a steady 1.5-3% faster
// than 256-lane workgroups.
// A 1024-lane workgroup allows 128 VGPRs per lane: the 8-neuron bf16 forward with spikes
// in the I/O dtype needs about 150 and spills some 40, yet still ran 2% / 5% faster than
// the spill-free 256-lane kernel at T = 64 / 256 (N = 2^24), so it keeps these workgroups.
constexpr int kSyncBlock = 1024;
constexpr int kSyncBf16Chunks = 6;

inline Plan make_plan(const snn_lif_cfg* c, int64_t T, int64_t N) {
    Plan p;
    // 2 neurons per lane (fp32 8-byte rows: 4 per lane measured 1% slower on large layers;
    // bf16 4-byte rows with 32-step chunks: faster than 4 per lane with 16-step chunks),
    // except bf16 layers of at most 16 steps that fill the chip: 4 per lane, 8-byte rows
    p.vb = N % 2 != 0 ? 1 : 2;
    if (c->io == SNN_IO_BF16 && T <= 16 && N % 4 == 0 && N / 4 >= kFillLanes) p.vb = 4;
    p.pipe = T > chunk_steps(p.vb) && N / p.vb < 4 * kFillLanes;
    p.k = chunk_steps(p.vb);
    if (!p.pipe && c->io == SNN_IO_BF16 && p.vb == 2) p.k = 32;
    if (T <= p.k) {
        for (int k : kShortChunks) {
            if (T <= k && k < p.k) {
                p.k = k;
                break;
            }
        }
    }
    // bf16 forward: 8 neurons per lane (16-byte rows, whole spike bytes) on large layers
    p.vf = (c->io == SNN_IO_BF16 && N % 8 == 0 && N / 8 >= kFillLanes) ? 8 : p.vb;
    const bool long_walk = !p.pipe && T > p.k;   // several chunks, not double-buffered
    p.blkf = long_walk && p.vf >= 2 ? kSyncBlock : kBlock;   // the lane widths measured
    p.blkb = long_walk && p.vb == 2 ? kSyncBlock : kBlock;
    p.syncb = c->io == SNN_IO_F32 || (T + p.k - 1) / p.k <= kSyncBf16Chunks;
    p.row_bytes = spike_row_bytes(c, N);
    const int64_t covered = c->spk == SNN_SPK_BITS ? p.row_bytes * 8 : N;
    p.lanes = (covered + p.vf - 1) / p.vf;
    return p;
}

// The layer fed by the previous layer's spikes reads one spike word per lane and row (2-8
// bytes) where the dense layer reads an I/O row of 8-16 bytes, so double-buffering its
// chunks costs more in occupancy than it hides (fp32 backward: 191 instead of 79 VGPRs, 2
// instead of 6 waves per SIMD; forward 127 instead of 69).  Its chunks are single-buffered
// at the dense layer's chunk length, so the checkpoint layout and snn_lif_saved_bytes stay
// the dense layer's.  At N = 2^19 (event timing, three alternating rounds): fp32 u8 spikes,
// T = 32: forward 10.2 instead of 10.5 us, backward 29.7-29.9 instead of 30.7-31.0 us; bf16
// bit spikes, T = 32: 11.1 instead of 11.8 us and 18.6 instead of 19.6-19.8 us; bf16 u8,
// T = 64: backward 32.8 instead of 35.7-36.0 us, forward within 1%.
inline Plan make_gain_plan(const snn_lif_cfg* c, int64_t T, int64_t N) {
    Plan p = make_plan(c, T, N);
    p.pipe = false;
    return p;
}

// A stack of L layers fused across depth (lif_stack_*_kernel): 16-step chunks -- L
// membranes per neuron and step in the backward's VGPRs -- or the shortest of kShortChunks
// that holds a short layer.  One neuron per lane on layers of up to kStackNarrowN neurons:
// the 3-layer backward then needs 77 VGPRs instead of 151, twice the waves hide the
// latency of its load-then-compute chunks, and it ran 5-13% faster than with 2 neurons per
// lane at 2^18-2^20 neurons (x[32][B*4096], B = 64-256; 2 layers 2-7%; below 2^18 the two
// are within the run-to-run spread); beyond that the 8-byte rows of 2 neurons per lane (1
// when N is odd) are as fast or faster (B = 768-2048).
constexpr int kMaxStackLayers = 3;
constexpr int64_t kStackNarrowN = 4 * kFillLanes;

struct StackPlan {
    int v;
    int k;
    int64_t lanes;
    int64_t row_bytes;
};

inline StackPlan make_stack_plan(const snn_lif_cfg* c, int64_t T, int64_t N) {
    StackPlan p;
    p.v = N % 2 != 0 || N <= kStackNarrowN ? 1 : 2;
    p.k = 16;
    for (int k : kShortChunks) {
        if (T <= k && k < p.k) {
            p.k = k;
            break;
        }
    }
    p.row_bytes = spike_row_bytes(c, N);
    const int64_t covered = c->spk == SNN_SPK_BITS ? p.row_bytes * 8 : N;
    p.lanes = (covered + p.v - 1) / p.v;
    return p;
}

inline int64_t stack_saved_bytes(const StackPlan& p, int L, int64_t T, int64_t N) {
    const int64_t chunks = (T + p.k - 1) / p.k;
    return chunks > 1 ? (chunks - 1) * L * N * int64_t(sizeof(float)) : 0;
}

inline int64_t saved_bytes(const Plan& p, int64_t T, int64_t N) {
    const int64_t chunks = (T + p.k - 1) / p.k;
    return chunks > 1 ? (chunks - 1) * N * int64_t(sizeof(float)) : 0;
}

inline LifK kernel_consts(const snn_lif_cfg* c) {
    LifK k;
    k.k = c->decay;
    k.th = c->v_th;
    k.rest = c->v_reset;
    k.alpha = c->alpha;
    k.c_exp = float(-double(c->alpha) * 1.4426950408889634074);  // -alpha log2(e)
    k.kth = c->decay * c->v_th;
    return k;
}

inline dim3 grid_for(int64_t lanes, int blk = kBlock) { return dim3(unsigned((lanes + blk - 1) / blk)); }

template <typename Tuple, size_t... I>
void fill_argv(Tuple& t, void** argv, std::index_sequence<I...>) {
    ((argv[I] = static_cast<void*>(&std::get<I>(t))), ...);
}

// Launch through hipLaunchKernel so the runtime's verdict is returned directly and the
// caller's sticky error state is left alone.
template <typename... P, typename... A>
snn_status launch_blk(void (*kernel)(P...), dim3 grid, int blk, hipStream_t stream, A... a) {
    static_assert(sizeof...(P) == sizeof...(A), "argument count");
    std::tuple<P...> args(a...);
    void* argv[sizeof...(P)];
    fill_argv(args, argv, std::index_sequence_for<P...>{});
    const hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(kernel), grid, dim3(blk), argv, 0, stream);
    return e == hipSuccess ? SNN_OK : SNN_E_LAUNCH;
}

template <typename... P, typename... A>
snn_status launch(void (*kernel)(P...), dim3 grid, hipStream_t stream, A... a) {
    return launch_blk(kernel, grid, kBlock, stream, a...);
}

// Rows per load batch of the forward.  The forward never revisits a row, so it need not
// hold a whole 32-step chunk (the checkpoint interval) in registers: it loads 16 rows at a
// time and checkpoints after every second batch.
constexpr int forward_batch(int io, int v, int k, bool pipe) {
    return (!pipe && k > 16) ? 16 : k;
}

// Calls f(V, K, PIPE) -- std::integral_constant / bool_constant tags -- with the lane width
// and chunk length the plan chose for the forward (vf) or the backward (vb): the
// combinations a kernel translation unit instantiates.
template <int I>
using IntC = std::integral_constant<int, I>;

template <int IO, int V, typename F>
snn_status chunk_variant(const Plan& p, F&& f) {
    constexpr int K = chunk_steps(V == 8 ? 2 : V);   // a double-buffered 8-wide lane would pair with 2-wide
    if (p.pipe) {
        if (p.k != K) return SNN_E_UNSUPPORTED;   // no plan pairs another chunk with these lanes
        return f(IntC<V>{}, IntC<K>{}, std::true_type{});
    }
    switch (p.k) {   // the long chunks, and the single-chunk layers of kShortChunks
        case 4: return f(IntC<V>{}, IntC<4>{}, std::false_type{});
        case 8: return f(IntC<V>{}, IntC<8>{}, std::false_type{});
        case 16: return f(IntC<V>{}, IntC<16>{}, std::false_type{});
        case 32: if constexpr (V == 1 || (IO == SNN_IO_BF16 && V != 4)) return f(IntC<V>{}, IntC<32>{}, std::false_type{});
                 break;
    }
    return SNN_E_UNSUPPORTED;
}

// Lane widths: 2 or 1; bf16 also 4 (short layers) and 8 (the forward of large layers).
template <int IO, typename F>
snn_status forward_variant(const Plan& p, F&& f) {
    switch (p.vf) {
        case 8: if constexpr (IO == SNN_IO_BF16) return chunk_variant<IO, 8>(p, f); break;
        case 4: if constexpr (IO == SNN_IO_BF16) return chunk_variant<IO, 4>(p, f); break;
        case 2: return chunk_variant<IO, 2>(p, f);
        case 1: return chunk_variant<IO, 1>(p, f);
    }
    return SNN_E_UNSUPPORTED;
}

template <int IO, typename F>
snn_status backward_variant(const Plan& p, F&& f) {
    switch (p.vb) {
        case 4: if constexpr (IO == SNN_IO_BF16) return chunk_variant<IO, 4>(p, f); break;
        case 2: return chunk_variant<IO, 2>(p, f);
        case 1: return chunk_variant<IO, 1>(p, f);
    }
    return SNN_E_UNSUPPORTED;
}

// v_in / v_last / g_in / g_out: the segment state of a sequence split along time (each may
// be null; see snn_lif_forward_seg and snn_lif_backward_seg).
template <int IO, int SPK>
snn_status forward_entry(int reset, const Plan& p, const LifK& k, int64_t T, int64_t N, const void* x,
                         void* spikes, void* saved, float* v_out, const float* v_in, float* v_last,
                         hipStream_t s);

template <int IO>
snn_status backward_entry(int reset, const Plan& p, const LifK& k, int64_t T, int64_t N, const void* x,
                          const void* saved, const void* gs, void* gx, const float* v_in, const float* g_in,
                          float* g_out, hipStream_t s);

// The layer fed by the previous layer's spikes (format SPK, u8 or bits) through a per-feature
// gain of F features.
template <int IO, int SPK>
snn_status forward_gain_entry(int reset, const Plan& p, const LifK& k, int64_t T, int64_t N, int64_t F,
                              const void* spikes_in, const float* gain, void* spikes, void* saved, float* v_out,
                              hipStream_t s);

template <int IO, int SPK>
snn_status backward_gain_entry(int reset, const Plan& p, const LifK& k, int64_t T, int64_t N, int64_t F,
                               const void* spikes_in, const float* gain, const void* saved, const void* gs,
                               void* gs_in, hipStream_t s);

// The stack fused across depth: gains is [L-1][F]; hidden and v_out may be null.
template <int IO, int SPK>
snn_status stack_forward_entry(int reset, int L, const StackPlan& p, const LifK& k, int64_t T, int64_t N, int64_t F,
                               const void* x, const float* gains, void* spikes, void* hidden, void* saved,
                               float* v_out, hipStream_t s);

template <int IO>
snn_status stack_backward_entry(int reset, int L, const StackPlan& p, const LifK& k, int64_t T, int64_t N, int64_t F,
                                const void* x, const float* gains, const void* saved, const void* gs, void* gx,
                                hipStream_t s);

snn_status gain_forward_entry(const snn_lif_cfg* c, int64_t T, int64_t N, int64_t F, const void* spikes,
                              int64_t row_bytes, const float* gain, void* x_next, hipStream_t s);

snn_status gain_backward_entry(const snn_lif_cfg* c, int64_t T, int64_t N, int64_t F, const void* gx_next,
                               const float* gain, void* gs, hipStream_t s);

snn_status serial_forward_entry(const snn_lif_cfg* c, const LifK& k, int64_t N, const void* x_t,
                                const float* v_prev, float* v_t, void* spikes_t, hipStream_t s);

snn_status serial_backward_entry(const snn_lif_cfg* c, const LifK& k, int64_t N, const float* v_t, const void* gs_t,
                                 const float* g_next, void* gx_t, float* g_out, hipStream_t s);

}  // namespace snnlif
