// Temporally fused LIF layer for MI355X (gfx950): forward and backward kernels and the
// C ABI declared in include/snn_lif.h.
//
// Design (see the header for the operation itself):
//  * Neurons are independent (Sec. 3.1), so each lane owns V consecutive neurons and walks
//    all T steps with their membranes in VGPRs (temporal fusion, Sec. 3.2).  Rows of the
//    time-major [T][N] tensors are read and written coalesced along N, 16 bytes per lane
//    (V = 4 fp32 or V = 8 bf16 neurons) when N is a multiple of V; otherwise V = 1.
//  * Time is processed in chunks of K steps.  All K input rows of a chunk are loaded before
//    the first step of the chunk is computed (they do not depend on the recurrence), so
//    every lane keeps K loads in flight.
//  * The forward saves no membrane for the backward except one fp32 checkpoint per neuron at
//    the end of every chunk but the last.  The backward walks the chunks in reverse: it
//    reloads the chunk's inputs, recomputes the chunk's membranes into VGPRs from the
//    checkpoint with the same instruction sequence as the forward (bit-identical), then
//    runs the reverse-time surrogate recurrence of Eq. (3) over the chunk.
//  * The membrane update is one IEEE multiply and one IEEE add (no fused multiply-add:
//    this file is compiled with -ffp-contract=off), so results are reproducible
//    bit for bit.  The backward uses fused multiply-adds where it wants them, explicitly.
//  * No MFMA: the work is elementwise across neurons and a scalar recurrence in time.
#include <hip/hip_runtime.h>

#include <climits>
#include <cmath>
#include <cstdint>
#include <tuple>
#include <type_traits>
#include <utility>

#include "snn_lif.h"

namespace {

constexpr int kBlock = 256;  // 4 wave64 per workgroup
constexpr int kWave = 64;

constexpr int64_t kMaxT = INT32_MAX;
constexpr int64_t kMaxN = int64_t(1) << 31;
constexpr int64_t kMaxTN = int64_t(1) << 44;

// Kernel-side hyper-parameters.
struct LifK {
    float k;      // decay k_tau
    float th;     // V_th
    float rest;   // V_rest
    float alpha;  // surrogate sharpness
    float c_exp;  // -alpha * log2(e): e^{-alpha |u|} = 2^{c_exp |u|}
    float kth;    // k * V_th (soft-reset backward)
};

// ------------------------------------------------------------------------------------
// Streaming memory access.  Every tensor element is touched once per kernel, so loads
// and stores carry the non-temporal hint.
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

template <typename E>
__device__ __forceinline__ E ld_nt(const void* p) {
    return __builtin_nontemporal_load(static_cast<const E*>(p));
}

template <typename E>
__device__ __forceinline__ void st_nt(void* p, E v) {
    __builtin_nontemporal_store(v, static_cast<E*>(p));
}

// Workgroups are dispatched round-robin over the 8 XCDs (workgroup b runs on XCD b % 8).
// Renumber them so that each XCD walks one contiguous range of the neuron axis: with the
// 32 MiB-apart rows of a [T][N] walk, this keeps each XCD's concurrent accesses local.
constexpr unsigned kXcds = 8;

__device__ __forceinline__ int64_t xcd_contiguous_block() {
    const unsigned nb = gridDim.x, b = blockIdx.x;
    const unsigned xcd = b % kXcds, slot = b / kXcds, q = nb / kXcds, r = nb % kXcds;
    return int64_t(xcd) * q + (xcd < r ? xcd : r) + slot;
}

// ------------------------------------------------------------------------------------
// Vectors of V consecutive neurons in the I/O dtype.
template <int IO, int V>
struct IoVec;

template <>
struct IoVec<SNN_IO_F32, 4> {
    using raw = f32x4_t;
    __device__ static raw load(const void* b, int64_t i) { return ld_nt<raw>(static_cast<const float*>(b) + i); }
    __device__ static float get(const raw& r, int j) { return r[j]; }
    __device__ static void store(void* b, int64_t i, const float (&f)[4]) {
        const raw v = {f[0], f[1], f[2], f[3]};
        st_nt(static_cast<float*>(b) + i, v);
    }
};

template <>
struct IoVec<SNN_IO_F32, 2> {
    using raw = f32x2_t;
    __device__ static raw load(const void* b, int64_t i) { return ld_nt<raw>(static_cast<const float*>(b) + i); }
    __device__ static float get(const raw& r, int j) { return r[j]; }
    __device__ static void store(void* b, int64_t i, const float (&f)[2]) {
        const raw v = {f[0], f[1]};
        st_nt(static_cast<float*>(b) + i, v);
    }
};

template <>
struct IoVec<SNN_IO_F32, 1> {
    using raw = float;
    __device__ static raw load(const void* b, int64_t i) { return ld_nt<raw>(static_cast<const float*>(b) + i); }
    __device__ static float get(const raw& r, int) { return r; }
    __device__ static void store(void* b, int64_t i, const float (&f)[1]) { st_nt(static_cast<float*>(b) + i, f[0]); }
};

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Two floats -> two bf16 (round to nearest even) packed low/high in one dword.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    f32x2_t v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

template <>
struct IoVec<SNN_IO_BF16, 8> {
    using raw = u32x4_t;
    __device__ static raw load(const void* b, int64_t i) { return ld_nt<raw>(static_cast<const uint16_t*>(b) + i); }
    __device__ static float get(const raw& r, int j) { return (j & 1) ? bf16_hi(r[j >> 1]) : bf16_lo(r[j >> 1]); }
    __device__ static void store(void* b, int64_t i, const float (&f)[8]) {
        const raw w = {pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]), pack_bf16x2(f[4], f[5]),
                       pack_bf16x2(f[6], f[7])};
        st_nt(static_cast<uint16_t*>(b) + i, w);
    }
};

template <>
struct IoVec<SNN_IO_BF16, 4> {
    using raw = u32x2_t;
    __device__ static raw load(const void* b, int64_t i) { return ld_nt<raw>(static_cast<const uint16_t*>(b) + i); }
    __device__ static float get(const raw& r, int j) { return (j & 1) ? bf16_hi(r[j >> 1]) : bf16_lo(r[j >> 1]); }
    __device__ static void store(void* b, int64_t i, const float (&f)[4]) {
        const raw w = {pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3])};
        st_nt(static_cast<uint16_t*>(b) + i, w);
    }
};

template <>
struct IoVec<SNN_IO_BF16, 2> {
    using raw = uint32_t;
    __device__ static raw load(const void* b, int64_t i) { return ld_nt<raw>(static_cast<const uint16_t*>(b) + i); }
    __device__ static float get(const raw& r, int j) { return j ? bf16_hi(r) : bf16_lo(r); }
    __device__ static void store(void* b, int64_t i, const float (&f)[2]) {
        st_nt(static_cast<uint16_t*>(b) + i, pack_bf16x2(f[0], f[1]));
    }
};

template <>
struct IoVec<SNN_IO_BF16, 1> {
    using raw = uint16_t;
    __device__ static raw load(const void* b, int64_t i) { return ld_nt<raw>(static_cast<const uint16_t*>(b) + i); }
    __device__ static float get(const raw& r, int) { return __uint_as_float(uint32_t(r) << 16); }
    __device__ static void store(void* b, int64_t i, const float (&f)[1]) {
        st_nt(static_cast<uint16_t*>(b) + i, static_cast<uint16_t>(pack_bf16x2(f[0], 0.0f) & 0xffffu));
    }
};

// ------------------------------------------------------------------------------------
// One step of Eq. (1) then Eq. (2) for one neuron.  `y` is the previous step's spike on
// entry and this step's on exit; `v` likewise for the membrane.
template <int RESET>
__device__ __forceinline__ void lif_step(const LifK& c, float& v, bool& y, float x) {
#pragma clang fp contract(off)
    if (RESET == SNN_RESET_HARD) {
        v = y ? c.rest + x : c.k * v + x;
    } else {
        const float w = y ? v - c.th : v;
        v = c.k * w + x;
    }
    y = v >= c.th;  // H(v - V_th) with H(0) = 1; NaN never fires
}

// Derivative of sigmoid(alpha u): alpha e / (1 + e)^2 with e = e^{-alpha |u|} (even in u).
__device__ __forceinline__ float surrogate(const LifK& c, float u) {
    const float e = __builtin_amdgcn_exp2f(c.c_exp * fabsf(u));
    const float r = __builtin_amdgcn_rcpf(1.0f + e);
    return (c.alpha * e) * (r * r);
}

// ------------------------------------------------------------------------------------
// Spike rows.  `t` is the row; lanes own neurons [n0, n0 + V).  A wave's share of a spike
// row can be less than a cache line (bits, or one byte per lane), so spikes are written
// with ordinary stores: the L2 merges the partial lines of neighbouring waves before they
// reach HBM, and a following kernel that reads the spikes can find them in cache.
template <int SPK, int V>
struct SpikeOut;

template <>
struct SpikeOut<SNN_SPK_U8, 4> {
    __device__ static void store(uint8_t* s, int64_t row_bytes, int64_t t, int64_t n0, bool active,
                                 const bool (&y)[4]) {
        const uint32_t w = uint32_t(y[0]) | (uint32_t(y[1]) << 8) | (uint32_t(y[2]) << 16) |
                           (uint32_t(y[3]) << 24);
        if (active) *reinterpret_cast<uint32_t*>(s + t * row_bytes + n0) = w;
    }
};

template <>
struct SpikeOut<SNN_SPK_U8, 8> {
    __device__ static void store(uint8_t* s, int64_t row_bytes, int64_t t, int64_t n0, bool active,
                                 const bool (&y)[8]) {
        uint2 w;
        w.x = uint32_t(y[0]) | (uint32_t(y[1]) << 8) | (uint32_t(y[2]) << 16) | (uint32_t(y[3]) << 24);
        w.y = uint32_t(y[4]) | (uint32_t(y[5]) << 8) | (uint32_t(y[6]) << 16) | (uint32_t(y[7]) << 24);
        if (active) *reinterpret_cast<uint2*>(s + t * row_bytes + n0) = w;
    }
};

template <>
struct SpikeOut<SNN_SPK_U8, 2> {
    __device__ static void store(uint8_t* s, int64_t row_bytes, int64_t t, int64_t n0, bool active,
                                 const bool (&y)[2]) {
        if (active) *reinterpret_cast<uint16_t*>(s + t * row_bytes + n0) = (uint16_t(uint32_t(y[0]) | (uint32_t(y[1]) << 8)));
    }
};

template <>
struct SpikeOut<SNN_SPK_U8, 1> {
    __device__ static void store(uint8_t* s, int64_t row_bytes, int64_t t, int64_t n0, bool active,
                                 const bool (&y)[1]) {
        if (active) s[t * row_bytes + n0] = uint8_t(y[0]);
    }
};

// Bits, 4 neurons per lane: lanes 2j and 2j+1 share a byte; the odd lane's nibble is
// moved to the even lane with a DPP quad permutation [1,0,3,2].  Every lane of the wave
// executes this (no divergence around it).
template <>
struct SpikeOut<SNN_SPK_BITS, 4> {
    __device__ static void store(uint8_t* s, int64_t row_bytes, int64_t t, int64_t n0, bool active,
                                 const bool (&y)[4]) {
        const int nib = active ? (int(y[0]) | (int(y[1]) << 1) | (int(y[2]) << 2) | (int(y[3]) << 3)) : 0;
        const int other = __builtin_amdgcn_mov_dpp(nib, 0xB1, 0xF, 0xF, false);
        if (((n0 >> 2) & 1) == 0 && n0 < row_bytes * 8)
            s[t * row_bytes + (n0 >> 3)] = uint8_t(nib | (other << 4));
    }
};

// Bits, 2 neurons per lane: four lanes share a byte; two DPP quad permutations ([1,0,3,2]
// then [2,3,0,1]) gather it in the first lane of each quad.
template <>
struct SpikeOut<SNN_SPK_BITS, 2> {
    __device__ static void store(uint8_t* s, int64_t row_bytes, int64_t t, int64_t n0, bool active,
                                 const bool (&y)[2]) {
        int b = active ? (int(y[0]) | (int(y[1]) << 1)) : 0;
        b |= __builtin_amdgcn_mov_dpp(b, 0xB1, 0xF, 0xF, false) << 2;
        b |= __builtin_amdgcn_mov_dpp(b, 0x4E, 0xF, 0xF, false) << 4;
        if (((n0 >> 1) & 3) == 0 && n0 < row_bytes * 8) s[t * row_bytes + (n0 >> 3)] = uint8_t(b);
    }
};

// Bits, 8 neurons per lane: each lane owns one byte of the row.
template <>
struct SpikeOut<SNN_SPK_BITS, 8> {
    __device__ static void store(uint8_t* s, int64_t row_bytes, int64_t t, int64_t n0, bool active,
                                 const bool (&y)[8]) {
        uint32_t b = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j) b |= uint32_t(y[j]) << j;
        if (n0 < row_bytes * 8) s[t * row_bytes + (n0 >> 3)] = uint8_t(active ? b : 0u);
    }
};

// Bits, 1 neuron per lane: one wave64 ballot is one 64-bit word of the row.
template <>
struct SpikeOut<SNN_SPK_BITS, 1> {
    __device__ static void store(uint8_t* s, int64_t row_bytes, int64_t t, int64_t n0, bool active,
                                 const bool (&y)[1]) {
        const uint64_t word = __ballot(active && y[0]);
        if ((threadIdx.x & (kWave - 1)) == 0 && n0 < row_bytes * 8)
            *reinterpret_cast<uint64_t*>(s + t * row_bytes + (n0 >> 3)) = word;
    }
};

// ------------------------------------------------------------------------------------
// fp32 rows of V neurons (checkpoints and the optional membrane output).
template <int V>
__device__ __forceinline__ void store_f32(float* p, const float (&f)[V]) {
    if constexpr (V == 8) {
        const f32x4_t lo = {f[0], f[1], f[2], f[3]}, hi = {f[4], f[5], f[6], f[7]};
        st_nt(p, lo);
        st_nt(p + 4, hi);
    } else if constexpr (V == 4) {
        const f32x4_t v = {f[0], f[1], f[2], f[3]};
        st_nt(p, v);
    } else if constexpr (V == 2) {
        const f32x2_t v = {f[0], f[1]};
        st_nt(p, v);
    } else {
        st_nt(p, f[0]);
    }
}

template <int V>
__device__ __forceinline__ void load_f32(const float* p, float (&f)[V]) {
    if constexpr (V == 4) {
        const f32x4_t a = ld_nt<f32x4_t>(p);
        f[0] = a[0];
        f[1] = a[1];
        f[2] = a[2];
        f[3] = a[3];
    } else if constexpr (V == 2) {
        const f32x2_t a = ld_nt<f32x2_t>(p);
        f[0] = a[0];
        f[1] = a[1];
    } else {
        f[0] = ld_nt<float>(p);
    }
}

// ------------------------------------------------------------------------------------
// Forward and backward bodies.  A chunk is K consecutive steps; only the last chunk of a
// layer can be shorter (T % K rows).  Row loads of a chunk are issued together, before the
// chunk's recurrence, because they do not depend on it.
//
// On gfx9-family GPUs one in-order counter (vmcnt) covers every outstanding vector load
// AND store, and the compiler's wait before a use is only as precise as the control flow
// allows: a load or store under a branch makes the merged count conservative, and then a
// wait for an old row also waits for younger loads.  So: workgroups whose lanes are all in
// range run a path with no per-lane guards (ALL = true), checkpoint loads are issued before
// the row loads they precede in use, and double-buffered loops peel their first iteration
// so that the loop body issues every load unconditionally.
template <int IO, int V, int K, bool FULL, bool REV>
__device__ __forceinline__ void load_rows(typename IoVec<IO, V>::raw (&buf)[K], const void* src, int64_t N,
                                          int64_t t0, int kn, int64_t n0) {
    using Io = IoVec<IO, V>;
    if constexpr (REV) {
#pragma unroll
        for (int i = K - 1; i >= 0; --i)
            if (FULL || i < kn) buf[i] = Io::load(src, (t0 + i) * N + n0);
    } else {
#pragma unroll
        for (int i = 0; i < K; ++i)
            if (FULL || i < kn) buf[i] = Io::load(src, (t0 + i) * N + n0);
    }
}

template <int IO, int SPK, int RESET, int V, int K, bool VOUT, bool FULL, bool ALL>
__device__ __forceinline__ void forward_rows(const LifK& c, const typename IoVec<IO, V>::raw (&xr)[K], int64_t N,
                                             int64_t t0, int kn, int64_t n0, bool active,
                                             uint8_t* __restrict__ spikes, int64_t row_bytes,
                                             float* __restrict__ v_out, float (&v)[V], bool (&y)[V]) {
    using Io = IoVec<IO, V>;
    const bool on = ALL || active;
#pragma unroll
    for (int i = 0; i < K; ++i) {
        if (FULL || i < kn) {
#pragma unroll
            for (int j = 0; j < V; ++j) lif_step<RESET>(c, v[j], y[j], on ? Io::get(xr[i], j) : 0.0f);
            SpikeOut<SPK, V>::store(spikes, row_bytes, t0 + i, n0, on, y);
            if (VOUT && on) store_f32<V>(v_out + (t0 + i) * N + n0, v);
        }
    }
}

// Forward of one workgroup's lanes.  Chunks 0 .. n_full-1 have K steps; a tail chunk of
// T % K steps follows when T % K != 0.  After every chunk but the last the membrane is
// checkpointed to saved[chunk][N].  PIPE: double-buffered chunks -- the next chunk's rows
// are in flight while the current chunk is computed (for layers with few lanes, where
// occupancy alone cannot hide the memory latency).
template <int IO, int SPK, int RESET, int V, int K, bool VOUT, bool PIPE, bool ALL>
__device__ __forceinline__ void forward_lanes(const LifK& c, int64_t T, int64_t N, int64_t n0,
                                              const void* __restrict__ x, uint8_t* __restrict__ spikes,
                                              int64_t row_bytes, float* __restrict__ saved,
                                              float* __restrict__ v_out) {
    using raw = typename IoVec<IO, V>::raw;
    const bool active = ALL || n0 < N;
    float v[V];
    bool y[V];
#pragma unroll
    for (int j = 0; j < V; ++j) {
        v[j] = c.rest;  // v^0 = V_rest
        y[j] = false;   // no spike before the first step
    }
    const int64_t n_full = T / K;
    const int k_tail = int(T % K);
    const int64_t last = k_tail ? n_full : n_full - 1;   // index of the last chunk
    // The scheduler must not move a chunk's compute across the batch of loads that
    // precedes it: that would change the outstanding-operation count between loop entry
    // and back-edge and make the compiler's waits conservative.
    auto load = [&](raw (&buf)[K], int64_t ch) {
        __builtin_amdgcn_sched_barrier(0);
        if (ALL || active) load_rows<IO, V, K, true, false>(buf, x, N, ch * K, K, n0);
        __builtin_amdgcn_sched_barrier(0);
    };
    // CKPT: 1 = this chunk is never the last (checkpoint unconditionally), 0 = test at run time
    auto step = [&](const raw (&buf)[K], int64_t ch, auto ckpt) {
        forward_rows<IO, SPK, RESET, V, K, VOUT, true, ALL>(c, buf, N, ch * K, K, n0, active, spikes, row_bytes,
                                                            v_out, v, y);
        if ((decltype(ckpt)::value || ch < last) && (ALL || active)) store_f32<V>(saved + ch * N + n0, v);
    };
    constexpr std::true_type not_last{};
    constexpr std::false_type maybe_last{};
    raw a[K];
    if constexpr (!PIPE) {
        for (int64_t ch = 0; ch < n_full; ++ch) {
            load(a, ch);
            step(a, ch, maybe_last);
        }
    } else if (n_full > 0) {
        raw b[K];
        load(a, 0);
        if (n_full == 1) {
            step(a, 0, maybe_last);
        } else {
            // Entering the loop, chunk ch is in flight in b and a is free: the same state
            // each iteration ends in, so the buffers keep their roles and every load and
            // store in the loop body is unconditional.
            load(b, 1);
            step(a, 0, not_last);
            int64_t ch = 1;
            for (; ch + 2 < n_full; ch += 2) {
                load(a, ch + 1);
                step(b, ch, not_last);
                load(b, ch + 2);
                step(a, ch + 1, not_last);
            }
            if (ch + 1 < n_full) {
                load(a, ch + 1);
                step(b, ch, not_last);
                step(a, ch + 1, maybe_last);
            } else {
                step(b, ch, maybe_last);
            }
        }
    }
    if (k_tail) {
        if (ALL || active) load_rows<IO, V, K, false, false>(a, x, N, n_full * K, k_tail, n0);
        forward_rows<IO, SPK, RESET, V, K, VOUT, false, ALL>(c, a, N, n_full * K, k_tail, n0, active, spikes,
                                                             row_bytes, v_out, v, y);
    }
}

// Grid: one lane per V neurons over ceil(max(N, 8*row_bytes) / V) lanes.  Lanes at or beyond
// N load nothing and report no spikes; they exist only to complete spike-bit words.
template <int IO, int SPK, int RESET, int V, int K, bool VOUT, bool PIPE>
__global__ __launch_bounds__(kBlock) void lif_forward_kernel(LifK c, int64_t T, int64_t N,
                                                             const void* __restrict__ x,
                                                             uint8_t* __restrict__ spikes,
                                                             int64_t row_bytes,
                                                             float* __restrict__ saved,
                                                             float* __restrict__ v_out) {
    const int64_t first = xcd_contiguous_block() * kBlock * V;
    const int64_t n0 = first + int64_t(threadIdx.x) * V;
    if (first + kBlock * V <= N)
        forward_lanes<IO, SPK, RESET, V, K, VOUT, PIPE, true>(c, T, N, n0, x, spikes, row_bytes, saved, v_out);
    else
        forward_lanes<IO, SPK, RESET, V, K, VOUT, PIPE, false>(c, T, N, n0, x, spikes, row_bytes, saved, v_out);
}

// Backward of one chunk.  v/y enter as the state before the chunk's first step; g enters
// as dL/dv of the step after the chunk and leaves as dL/dv of the chunk's first step.
template <int IO, int RESET, int V, int K, bool FULL>
__device__ __forceinline__ void backward_rows(const LifK& c, const typename IoVec<IO, V>::raw (&xr)[K],
                                              const typename IoVec<IO, V>::raw (&gr)[K], int64_t N, int64_t t0,
                                              int kn, int64_t n0, void* gx, float (&v)[V], bool (&y)[V],
                                              float (&g)[V]) {
    using Io = IoVec<IO, V>;
    // recompute the chunk's membranes, bit-identical to the forward
    float vs[K][V];
#pragma unroll
    for (int i = 0; i < K; ++i) {
        if (FULL || i < kn) {
#pragma unroll
            for (int j = 0; j < V; ++j) {
                lif_step<RESET>(c, v[j], y[j], Io::get(xr[i], j));
                vs[i][j] = v[j];
            }
        }
    }
    // Eq. (3) in reverse time: g^t = dL/dy^t delta^t + (dv^{t+1}/dv^t) g^{t+1}
#pragma unroll
    for (int i = K - 1; i >= 0; --i) {
        if (FULL || i < kn) {
            float out[V];
#pragma unroll
            for (int j = 0; j < V; ++j) {
                const float vt = vs[i][j];
                const float d = surrogate(c, vt - c.th);
                float dv_next;
                if (RESET == SNN_RESET_HARD)  // k (1 - y^t) + (V_rest - k v^t) delta^t
                    dv_next = fmaf(fmaf(-c.k, vt, c.rest), d, vt >= c.th ? 0.0f : c.k);
                else                          // k (1 - V_th delta^t)
                    dv_next = fmaf(-c.kth, d, c.k);
                g[j] = fmaf(Io::get(gr[i], j), d, dv_next * g[j]);
                out[j] = g[j];
            }
            Io::store(gx, (t0 + i) * N + n0, out);
        }
    }
}

// Everything the backward of chunk ch reads: the state entering it (loaded first), its
// input rows, and its dL/dy rows (issued last-first, the order the reverse pass uses them).
template <int IO, int V, int K>
struct BwdChunk {
    typename IoVec<IO, V>::raw x[K];
    typename IoVec<IO, V>::raw gs[K];
    float v[V];
};

// ALWAYS: the layer has a checkpoint row, so the state is loaded unconditionally (chunk 0
// reads row 0 and then takes V_rest instead), keeping the caller's loop free of branches.
template <int IO, int V, int K, bool FULL, bool ALWAYS>
__device__ __forceinline__ void backward_load(BwdChunk<IO, V, K>& b, const LifK& c, const void* __restrict__ x,
                                              const float* __restrict__ saved, const void* gs, int64_t N,
                                              int64_t ch, int kn, int64_t n0) {
    if (ALWAYS) {
        load_f32<V>(saved + (ch > 0 ? ch - 1 : 0) * N + n0, b.v);
    } else if (ch == 0) {
#pragma unroll
        for (int j = 0; j < V; ++j) b.v[j] = c.rest;
    } else {
        load_f32<V>(saved + (ch - 1) * N + n0, b.v);
    }
    load_rows<IO, V, K, FULL, false>(b.x, x, N, ch * K, kn, n0);
    load_rows<IO, V, K, FULL, true>(b.gs, gs, N, ch * K, kn, n0);
}

template <int IO, int RESET, int V, int K, bool FULL>
__device__ __forceinline__ void backward_chunk(const LifK& c, const BwdChunk<IO, V, K>& b, int64_t N, int64_t ch,
                                               int kn, int64_t n0, void* gx, float (&g)[V]) {
    float v[V];
    bool y[V];
#pragma unroll
    for (int j = 0; j < V; ++j) {
        v[j] = ch > 0 ? b.v[j] : c.rest;
        y[j] = ch > 0 && b.v[j] >= c.th;  // a checkpoint is a post-step membrane; step 0 has y = 0
    }
    backward_rows<IO, RESET, V, K, FULL>(c, b.x, b.gs, N, ch * K, kn, n0, gx, v, y, g);
}

// Chunks are processed last-first: the short tail chunk (if any), then the full chunks.
template <int IO, int RESET, int V, int K, bool PIPE>
__device__ __forceinline__ void backward_lanes(const LifK& c, int64_t T, int64_t N, int64_t n0,
                                               const void* __restrict__ x, const float* __restrict__ saved,
                                               const void* gs, void* gx) {
    float g[V];
#pragma unroll
    for (int j = 0; j < V; ++j) g[j] = 0.0f;  // dL/dv^{T+1} = 0
    const int64_t n_full = T / K;
    const int k_tail = int(T % K);
    BwdChunk<IO, V, K> a;
    if (k_tail) {
        backward_load<IO, V, K, false, false>(a, c, x, saved, gs, N, n_full, k_tail, n0);
        backward_chunk<IO, RESET, V, K, false>(c, a, N, n_full, k_tail, n0, gx, g);
    }
    auto load = [&](BwdChunk<IO, V, K>& buf, int64_t ch) {
        __builtin_amdgcn_sched_barrier(0);
        backward_load<IO, V, K, true, PIPE>(buf, c, x, saved, gs, N, ch, K, n0);
        __builtin_amdgcn_sched_barrier(0);
    };
    auto step = [&](const BwdChunk<IO, V, K>& buf, int64_t ch) {
        backward_chunk<IO, RESET, V, K, true>(c, buf, N, ch, K, n0, gx, g);
    };
    if constexpr (!PIPE) {
        for (int64_t ch = n_full - 1; ch >= 0; --ch) {
            load(a, ch);
            step(a, ch);
        }
    } else if (n_full > 0) {
        BwdChunk<IO, V, K> b;
        load(a, n_full - 1);
        if (n_full == 1) {
            step(a, 0);
        } else {
            // as in the forward: entering the loop, chunk ch is in flight in b, a is free
            load(b, n_full - 2);
            step(a, n_full - 1);
            int64_t ch = n_full - 2;
            for (; ch >= 2; ch -= 2) {
                load(a, ch - 1);
                step(b, ch);
                load(b, ch - 2);
                step(a, ch - 1);
            }
            if (ch >= 1) {
                load(a, ch - 1);
                step(b, ch);
                step(a, ch - 1);
            } else {
                step(b, ch);
            }
        }
    }
}

template <int IO, int RESET, int V, int K, bool PIPE>
__global__ __launch_bounds__(kBlock) void lif_backward_kernel(LifK c, int64_t T, int64_t N,
                                                              const void* __restrict__ x,
                                                              const float* __restrict__ saved,
                                                              const void* gs, void* gx) {
    const int64_t first = xcd_contiguous_block() * kBlock * V;
    const int64_t n0 = first + int64_t(threadIdx.x) * V;
    if (first + kBlock * V > N && n0 >= N) return;
    backward_lanes<IO, RESET, V, K, PIPE>(c, T, N, n0, x, saved, gs, gx);
}

// ------------------------------------------------------------------------------------
// Per-feature gain between stacked layers.  One lane per V neurons walks all T rows,
// kGlueRows rows of loads in flight at a time.
constexpr int kGlueRows = 8;

// The spike word holding a lane's V neurons of row t (u8: V bytes; bits: their byte).
template <int SPK, int V>
__device__ __forceinline__ uint32_t spike_word(const uint8_t* s, int64_t row_bytes, int64_t t, int64_t n0) {
    if constexpr (SPK == SNN_SPK_U8) {
        if constexpr (V == 4) return *reinterpret_cast<const uint32_t*>(s + t * row_bytes + n0);
        else return s[t * row_bytes + n0];
    } else {
        return s[t * row_bytes + (n0 >> 3)];
    }
}

template <int SPK, int V>
__device__ __forceinline__ float spike_of(uint32_t w, int64_t n0, int j) {
    if constexpr (SPK == SNN_SPK_U8) return float((w >> (8 * j)) & 0xffu);
    else return float((w >> ((n0 + j) & 7)) & 1u);
}

template <int IO, int SPK, int V>
__global__ __launch_bounds__(kBlock) void gain_forward_kernel(int64_t T, int64_t N, int64_t F,
                                                              const uint8_t* __restrict__ spikes,
                                                              int64_t row_bytes,
                                                              const float* __restrict__ gain,
                                                              void* __restrict__ x_next) {
    const int64_t n0 = (xcd_contiguous_block() * kBlock + threadIdx.x) * V;
    if (n0 >= N) return;
    float gv[V];
#pragma unroll
    for (int j = 0; j < V; ++j) gv[j] = gain[(n0 + j) % F];
    auto emit = [&](uint32_t w, int64_t t) {
        float out[V];
#pragma unroll
        for (int j = 0; j < V; ++j) out[j] = gv[j] * spike_of<SPK, V>(w, n0, j);
        IoVec<IO, V>::store(x_next, t * N + n0, out);
    };
    int64_t t0 = 0;
    for (; t0 + kGlueRows <= T; t0 += kGlueRows) {
        uint32_t w[kGlueRows];
#pragma unroll
        for (int i = 0; i < kGlueRows; ++i) w[i] = spike_word<SPK, V>(spikes, row_bytes, t0 + i, n0);
#pragma unroll
        for (int i = 0; i < kGlueRows; ++i) emit(w[i], t0 + i);
    }
    for (; t0 < T; ++t0) emit(spike_word<SPK, V>(spikes, row_bytes, t0, n0), t0);
}

template <int IO, int V>
__global__ __launch_bounds__(kBlock) void gain_backward_kernel(int64_t T, int64_t N, int64_t F,
                                                               const void* gx_next,
                                                               const float* __restrict__ gain,
                                                               void* gs) {
    using Io = IoVec<IO, V>;
    const int64_t n0 = (xcd_contiguous_block() * kBlock + threadIdx.x) * V;
    if (n0 >= N) return;
    float gv[V];
#pragma unroll
    for (int j = 0; j < V; ++j) gv[j] = gain[(n0 + j) % F];
    auto emit = [&](const typename Io::raw& r, int64_t t) {
        float out[V];
#pragma unroll
        for (int j = 0; j < V; ++j) out[j] = gv[j] * Io::get(r, j);
        Io::store(gs, t * N + n0, out);
    };
    int64_t t0 = 0;
    for (; t0 + kGlueRows <= T; t0 += kGlueRows) {
        typename Io::raw r[kGlueRows];
#pragma unroll
        for (int i = 0; i < kGlueRows; ++i) r[i] = Io::load(gx_next, (t0 + i) * N + n0);
#pragma unroll
        for (int i = 0; i < kGlueRows; ++i) emit(r[i], t0 + i);
    }
    for (; t0 < T; ++t0) emit(Io::load(gx_next, t0 * N + n0), t0);
}

// ------------------------------------------------------------------------------------
// Host side.

template <typename Tuple, size_t... I>
void fill_argv(Tuple& t, void** argv, std::index_sequence<I...>) {
    ((argv[I] = static_cast<void*>(&std::get<I>(t))), ...);
}

// Launch through hipLaunchKernel so the runtime's verdict is returned directly and the
// caller's sticky error state is left alone.
template <typename... P, typename... A>
snn_status launch(void (*kernel)(P...), dim3 grid, hipStream_t stream, A... a) {
    static_assert(sizeof...(P) == sizeof...(A), "argument count");
    std::tuple<P...> args(a...);
    void* argv[sizeof...(P)];
    fill_argv(args, argv, std::index_sequence_for<P...>{});
    const hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(kernel), grid, dim3(kBlock), argv, 0, stream);
    return e == hipSuccess ? SNN_OK : SNN_E_LAUNCH;
}

snn_status check_cfg(const snn_lif_cfg* c) {
    if (c == nullptr) return SNN_E_NULL;
    if (!(c->decay >= 0.0f && c->decay <= 1.0f)) return SNN_E_PARAM;  // also rejects NaN
    if (!std::isfinite(c->v_th) || !std::isfinite(c->v_reset)) return SNN_E_PARAM;
    if (!(c->alpha > 0.0f) || !std::isfinite(c->alpha)) return SNN_E_PARAM;
    if (c->reset != SNN_RESET_HARD && c->reset != SNN_RESET_SOFT) return SNN_E_PARAM;
    if (c->io != SNN_IO_F32 && c->io != SNN_IO_BF16) return SNN_E_PARAM;
    if (c->spk != SNN_SPK_U8 && c->spk != SNN_SPK_BITS) return SNN_E_PARAM;
    return SNN_OK;
}

snn_status check_shape(int64_t T, int64_t N) {
    if (T < 0 || N < 0 || T > kMaxT || N > kMaxN) return SNN_E_SHAPE;
    if (T > 0 && N > kMaxTN / T) return SNN_E_SHAPE;
    return SNN_OK;
}

bool aligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int64_t spike_row_bytes(const snn_lif_cfg* c, int64_t N) {
    return c->spk == SNN_SPK_U8 ? N : 8 * ((N + 63) / 64);
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
    int64_t lanes;   // lanes in the forward grid
    int64_t row_bytes;
};

// Steps per chunk: the backward keeps K membranes per neuron in VGPRs plus K rows of x and
// dL/dy (twice the rows when double-buffered); bf16 rows take half the registers.
constexpr int chunk_steps(int io, int v, bool pipe) {
    return v == 4 ? (pipe && io == SNN_IO_F32 ? 8 : 16) : v == 2 ? 16 : 32;
}

// Lanes that fill the chip with 16 waves per CU (256 CUs x 16 x 64).
constexpr int64_t kFillLanes = int64_t(256) * 16 * 64;

Plan make_plan(const snn_lif_cfg* c, int64_t T, int64_t N) {
    Plan p;
    p.vb = N % 4 == 0 ? 4 : N % 2 == 0 ? 2 : 1;
    if (p.vb == 4 && N / 4 < kFillLanes) p.vb = 2;   // twice the lanes for small layers
    p.pipe = T > chunk_steps(c->io, p.vb, false) && N / p.vb < 4 * kFillLanes;
    p.k = chunk_steps(c->io, p.vb, p.pipe);
    // bf16 forward: 8 neurons per lane (16-byte rows, whole spike bytes) on large layers
    p.vf = (c->io == SNN_IO_BF16 && p.vb == 4 && N % 8 == 0 && N / 8 >= kFillLanes) ? 8 : p.vb;
    p.row_bytes = spike_row_bytes(c, N);
    const int64_t covered = c->spk == SNN_SPK_BITS ? p.row_bytes * 8 : N;
    p.lanes = (covered + p.vf - 1) / p.vf;
    return p;
}

int64_t saved_bytes(const Plan& p, int64_t T, int64_t N) {
    const int64_t chunks = (T + p.k - 1) / p.k;
    return chunks > 1 ? (chunks - 1) * N * int64_t(sizeof(float)) : 0;
}

LifK kernel_consts(const snn_lif_cfg* c) {
    LifK k;
    k.k = c->decay;
    k.th = c->v_th;
    k.rest = c->v_reset;
    k.alpha = c->alpha;
    k.c_exp = float(-double(c->alpha) * 1.4426950408889634074);  // -alpha log2(e)
    k.kth = c->decay * c->v_th;
    return k;
}

dim3 grid_for(int64_t lanes) { return dim3(unsigned((lanes + kBlock - 1) / kBlock)); }

template <int IO, int SPK, int RESET, int V, int K, bool PIPE>
snn_status forward_launch_v(const Plan& p, const LifK& k, int64_t T, int64_t N, const void* x, uint8_t* sp,
                            float* sv, float* v_out, hipStream_t s) {
    const dim3 g = grid_for(p.lanes);
    return v_out ? launch(lif_forward_kernel<IO, SPK, RESET, V, K, true, PIPE>, g, s, k, T, N, x, sp, p.row_bytes, sv, v_out)
                 : launch(lif_forward_kernel<IO, SPK, RESET, V, K, false, PIPE>, g, s, k, T, N, x, sp, p.row_bytes, sv, v_out);
}

// (vf, vb, pipe) combinations the planner produces.
template <int IO, int SPK, int RESET>
snn_status forward_launch(const Plan& p, const LifK& k, int64_t T, int64_t N, const void* x, void* spikes,
                          void* saved, float* v_out, hipStream_t s) {
    uint8_t* sp = static_cast<uint8_t*>(spikes);
    float* sv = static_cast<float*>(saved);
    constexpr int K4 = chunk_steps(IO, 4, false), K4p = chunk_steps(IO, 4, true);
    constexpr int K2 = chunk_steps(IO, 2, false), K1 = chunk_steps(IO, 1, false);
    if constexpr (IO == SNN_IO_BF16) {
        if (p.vf == 8)
            return p.pipe ? forward_launch_v<IO, SPK, RESET, 8, K4p, true>(p, k, T, N, x, sp, sv, v_out, s)
                          : forward_launch_v<IO, SPK, RESET, 8, K4, false>(p, k, T, N, x, sp, sv, v_out, s);
    }
    switch (p.vf * 2 + int(p.pipe)) {
        case 8: return forward_launch_v<IO, SPK, RESET, 4, K4, false>(p, k, T, N, x, sp, sv, v_out, s);
        case 9: return forward_launch_v<IO, SPK, RESET, 4, K4p, true>(p, k, T, N, x, sp, sv, v_out, s);
        case 4: return forward_launch_v<IO, SPK, RESET, 2, K2, false>(p, k, T, N, x, sp, sv, v_out, s);
        case 5: return forward_launch_v<IO, SPK, RESET, 2, K2, true>(p, k, T, N, x, sp, sv, v_out, s);
        case 2: return forward_launch_v<IO, SPK, RESET, 1, K1, false>(p, k, T, N, x, sp, sv, v_out, s);
        default: return forward_launch_v<IO, SPK, RESET, 1, K1, true>(p, k, T, N, x, sp, sv, v_out, s);
    }
}

template <int IO, int RESET, int V, bool PIPE>
snn_status backward_launch_v(const LifK& k, int64_t T, int64_t N, const void* x, const float* sv, const void* gs,
                             void* gx, hipStream_t s) {
    constexpr int K = chunk_steps(IO, V, PIPE);
    return launch(lif_backward_kernel<IO, RESET, V, K, PIPE>, grid_for((N + V - 1) / V), s, k, T, N, x, sv, gs, gx);
}

template <int IO, int RESET>
snn_status backward_launch(const Plan& p, const LifK& k, int64_t T, int64_t N, const void* x,
                           const void* saved, const void* gs, void* gx, hipStream_t s) {
    const float* sv = static_cast<const float*>(saved);
    switch (p.vb * 2 + int(p.pipe)) {
        case 8: return backward_launch_v<IO, RESET, 4, false>(k, T, N, x, sv, gs, gx, s);
        case 9: return backward_launch_v<IO, RESET, 4, true>(k, T, N, x, sv, gs, gx, s);
        case 4: return backward_launch_v<IO, RESET, 2, false>(k, T, N, x, sv, gs, gx, s);
        case 5: return backward_launch_v<IO, RESET, 2, true>(k, T, N, x, sv, gs, gx, s);
        case 2: return backward_launch_v<IO, RESET, 1, false>(k, T, N, x, sv, gs, gx, s);
        default: return backward_launch_v<IO, RESET, 1, true>(k, T, N, x, sv, gs, gx, s);
    }
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

snn_status snn_lif_forward(const snn_lif_cfg* cfg, int64_t T, int64_t N, const void* x, void* spikes,
                           void* saved, float* v_out, void* stream) {
    snn_status st = check_cfg(cfg);
    if (st != SNN_OK) return st;
    if ((st = check_shape(T, N)) != SNN_OK) return st;
    if (T == 0 || N == 0) return SNN_OK;
    const Plan p = make_plan(cfg, T, N);
    const bool need_saved = saved_bytes(p, T, N) > 0;
    if (x == nullptr || spikes == nullptr || (need_saved && saved == nullptr)) return SNN_E_NULL;
    if (!aligned(x) || !aligned(spikes) || (saved && !aligned(saved)) || (v_out && !aligned(v_out)))
        return SNN_E_ALIGN;
    const LifK k = kernel_consts(cfg);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool bits = cfg->spk == SNN_SPK_BITS, soft = cfg->reset == SNN_RESET_SOFT;
    if (cfg->io == SNN_IO_F32) {
        if (bits)
            return soft ? forward_launch<SNN_IO_F32, SNN_SPK_BITS, SNN_RESET_SOFT>(p, k, T, N, x, spikes, saved, v_out, s)
                        : forward_launch<SNN_IO_F32, SNN_SPK_BITS, SNN_RESET_HARD>(p, k, T, N, x, spikes, saved, v_out, s);
        return soft ? forward_launch<SNN_IO_F32, SNN_SPK_U8, SNN_RESET_SOFT>(p, k, T, N, x, spikes, saved, v_out, s)
                    : forward_launch<SNN_IO_F32, SNN_SPK_U8, SNN_RESET_HARD>(p, k, T, N, x, spikes, saved, v_out, s);
    }
    if (bits)
        return soft ? forward_launch<SNN_IO_BF16, SNN_SPK_BITS, SNN_RESET_SOFT>(p, k, T, N, x, spikes, saved, v_out, s)
                    : forward_launch<SNN_IO_BF16, SNN_SPK_BITS, SNN_RESET_HARD>(p, k, T, N, x, spikes, saved, v_out, s);
    return soft ? forward_launch<SNN_IO_BF16, SNN_SPK_U8, SNN_RESET_SOFT>(p, k, T, N, x, spikes, saved, v_out, s)
                : forward_launch<SNN_IO_BF16, SNN_SPK_U8, SNN_RESET_HARD>(p, k, T, N, x, spikes, saved, v_out, s);
}

snn_status snn_lif_backward(const snn_lif_cfg* cfg, int64_t T, int64_t N, const void* x, const void* saved,
                            const void* grad_s, void* grad_x, void* stream) {
    snn_status st = check_cfg(cfg);
    if (st != SNN_OK) return st;
    if ((st = check_shape(T, N)) != SNN_OK) return st;
    if (T == 0 || N == 0) return SNN_OK;
    const Plan p = make_plan(cfg, T, N);
    const bool need_saved = saved_bytes(p, T, N) > 0;
    if (x == nullptr || grad_s == nullptr || grad_x == nullptr || (need_saved && saved == nullptr))
        return SNN_E_NULL;
    if (!aligned(x) || !aligned(grad_s) || !aligned(grad_x) || (saved && !aligned(saved))) return SNN_E_ALIGN;
    const LifK k = kernel_consts(cfg);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool soft = cfg->reset == SNN_RESET_SOFT;
    if (cfg->io == SNN_IO_F32)
        return soft ? backward_launch<SNN_IO_F32, SNN_RESET_SOFT>(p, k, T, N, x, saved, grad_s, grad_x, s)
                    : backward_launch<SNN_IO_F32, SNN_RESET_HARD>(p, k, T, N, x, saved, grad_s, grad_x, s);
    return soft ? backward_launch<SNN_IO_BF16, SNN_RESET_SOFT>(p, k, T, N, x, saved, grad_s, grad_x, s)
                : backward_launch<SNN_IO_BF16, SNN_RESET_HARD>(p, k, T, N, x, saved, grad_s, grad_x, s);
}

static snn_status check_gain_shape(int64_t T, int64_t B, int64_t F) {
    if (T < 0 || B < 0 || F < 0) return SNN_E_SHAPE;
    if (B > 0 && F > kMaxN / B) return SNN_E_SHAPE;
    return check_shape(T, B * F);
}

static dim3 gain_grid(int64_t lanes) { return grid_for(lanes); }

snn_status snn_gain_spikes_forward(const snn_lif_cfg* cfg, int64_t T, int64_t B, int64_t F, const void* spikes,
                                   const float* gain, void* x_next, void* stream) {
    snn_status st = check_cfg(cfg);
    if (st != SNN_OK) return st;
    if ((st = check_gain_shape(T, B, F)) != SNN_OK) return st;
    const int64_t N = B * F;
    if (T == 0 || N == 0) return SNN_OK;
    if (spikes == nullptr || gain == nullptr || x_next == nullptr) return SNN_E_NULL;
    if (!aligned(spikes) || !aligned(gain) || !aligned(x_next)) return SNN_E_ALIGN;
    const int64_t row = spike_row_bytes(cfg, N);
    const uint8_t* sp = static_cast<const uint8_t*>(spikes);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool v4 = N % 4 == 0;
    const dim3 grid = gain_grid(v4 ? N / 4 : N);
    const bool bits = cfg->spk == SNN_SPK_BITS;
    if (cfg->io == SNN_IO_F32) {
        if (v4)
            return bits ? launch(gain_forward_kernel<SNN_IO_F32, SNN_SPK_BITS, 4>, grid, s, T, N, F, sp, row, gain, x_next)
                        : launch(gain_forward_kernel<SNN_IO_F32, SNN_SPK_U8, 4>, grid, s, T, N, F, sp, row, gain, x_next);
        return bits ? launch(gain_forward_kernel<SNN_IO_F32, SNN_SPK_BITS, 1>, grid, s, T, N, F, sp, row, gain, x_next)
                    : launch(gain_forward_kernel<SNN_IO_F32, SNN_SPK_U8, 1>, grid, s, T, N, F, sp, row, gain, x_next);
    }
    if (v4)
        return bits ? launch(gain_forward_kernel<SNN_IO_BF16, SNN_SPK_BITS, 4>, grid, s, T, N, F, sp, row, gain, x_next)
                    : launch(gain_forward_kernel<SNN_IO_BF16, SNN_SPK_U8, 4>, grid, s, T, N, F, sp, row, gain, x_next);
    return bits ? launch(gain_forward_kernel<SNN_IO_BF16, SNN_SPK_BITS, 1>, grid, s, T, N, F, sp, row, gain, x_next)
                : launch(gain_forward_kernel<SNN_IO_BF16, SNN_SPK_U8, 1>, grid, s, T, N, F, sp, row, gain, x_next);
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
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool v4 = N % 4 == 0;
    const dim3 grid = gain_grid(v4 ? N / 4 : N);
    if (cfg->io == SNN_IO_F32)
        return v4 ? launch(gain_backward_kernel<SNN_IO_F32, 4>, grid, s, T, N, F, grad_x_next, gain, grad_s)
                  : launch(gain_backward_kernel<SNN_IO_F32, 1>, grid, s, T, N, F, grad_x_next, gain, grad_s);
    return v4 ? launch(gain_backward_kernel<SNN_IO_BF16, 4>, grid, s, T, N, F, grad_x_next, gain, grad_s)
              : launch(gain_backward_kernel<SNN_IO_BF16, 1>, grid, s, T, N, F, grad_x_next, gain, grad_s);
}

}  // extern "C"
