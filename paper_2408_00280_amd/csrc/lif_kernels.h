// Device code of the temporally fused LIF layer for MI355X (gfx950): forward and
// backward kernels and the stacked-layer gain kernels.  Each kernel translation unit
// includes this header and instantiates one slice of the kernel variants.
//
// Design (see the header for the operation itself):
//  * Neurons are independent (Sec. 3.1), so each lane owns V consecutive neurons and walks
//    all T steps with their membranes in VGPRs (temporal fusion, Sec. 3.2).  Rows of the
//    time-major [T][N] tensors are read and written coalesced along N, 8 or 16 bytes per
//    lane (V = 2 fp32, V = 4 or 8 bf16 neurons) when N is a multiple of V; otherwise fewer.
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
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "lif_common.h"

namespace snnlif {

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

// A float rounded to the I/O dtype (to nearest even for bf16), as a float.
template <int IO>
__device__ __forceinline__ float io_round(float f) {
    if constexpr (IO == SNN_IO_BF16) return bf16_lo(pack_bf16x2(f, 0.0f));
    else return f;
}

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
struct SpikeFmt;

template <>
struct SpikeFmt<SNN_SPK_U8, 4> {
    __device__ static void store(uint8_t* s, int64_t row_bytes, int64_t t, int64_t n0, bool active,
                                 const bool (&y)[4]) {
        const uint32_t w = uint32_t(y[0]) | (uint32_t(y[1]) << 8) | (uint32_t(y[2]) << 16) |
                           (uint32_t(y[3]) << 24);
        if (active) *reinterpret_cast<uint32_t*>(s + t * row_bytes + n0) = w;
    }
};

template <>
struct SpikeFmt<SNN_SPK_U8, 8> {
    __device__ static void store(uint8_t* s, int64_t row_bytes, int64_t t, int64_t n0, bool active,
                                 const bool (&y)[8]) {
        uint2 w;
        w.x = uint32_t(y[0]) | (uint32_t(y[1]) << 8) | (uint32_t(y[2]) << 16) | (uint32_t(y[3]) << 24);
        w.y = uint32_t(y[4]) | (uint32_t(y[5]) << 8) | (uint32_t(y[6]) << 16) | (uint32_t(y[7]) << 24);
        if (active) *reinterpret_cast<uint2*>(s + t * row_bytes + n0) = w;
    }
};

template <>
struct SpikeFmt<SNN_SPK_U8, 2> {
    __device__ static void store(uint8_t* s, int64_t row_bytes, int64_t t, int64_t n0, bool active,
                                 const bool (&y)[2]) {
        if (active) *reinterpret_cast<uint16_t*>(s + t * row_bytes + n0) = (uint16_t(uint32_t(y[0]) | (uint32_t(y[1]) << 8)));
    }
};

template <>
struct SpikeFmt<SNN_SPK_U8, 1> {
    __device__ static void store(uint8_t* s, int64_t row_bytes, int64_t t, int64_t n0, bool active,
                                 const bool (&y)[1]) {
        if (active) s[t * row_bytes + n0] = uint8_t(y[0]);
    }
};

// Bits, 4 neurons per lane: lanes 2j and 2j+1 share a byte; the odd lane's nibble is
// moved to the even lane with a DPP quad permutation [1,0,3,2].  Every lane of the wave
// executes this (no divergence around it).
template <>
struct SpikeFmt<SNN_SPK_BITS, 4> {
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
struct SpikeFmt<SNN_SPK_BITS, 2> {
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
struct SpikeFmt<SNN_SPK_BITS, 8> {
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
struct SpikeFmt<SNN_SPK_BITS, 1> {
    __device__ static void store(uint8_t* s, int64_t row_bytes, int64_t t, int64_t n0, bool active,
                                 const bool (&y)[1]) {
        const uint64_t word = __ballot(active && y[0]);
        if ((threadIdx.x & (kWave - 1)) == 0 && n0 < row_bytes * 8)
            *reinterpret_cast<uint64_t*>(s + t * row_bytes + (n0 >> 3)) = word;
    }
};

// Spikes as 0/1 values in the I/O dtype ([T][N] like x): ready for a following ANN
// operator.  Written through the streaming I/O path; rows are full cache lines.
template <int IO, int SPK, int V>
struct SpikeOut : SpikeFmt<SPK, V> {};

template <int IO, int V>
struct SpikeOut<IO, SNN_SPK_IO, V> {
    __device__ static void store(uint8_t* s, int64_t row_bytes, int64_t t, int64_t n0, bool active,
                                 const bool (&y)[V]) {
        constexpr int64_t esize = IO == SNN_IO_F32 ? 4 : 2;
        float f[V];
#pragma unroll
        for (int j = 0; j < V; ++j) f[j] = y[j] ? 1.0f : 0.0f;
        if (active) IoVec<IO, V>::store(s, t * (row_bytes / esize) + n0, f);
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
    if constexpr (V == 8) {
        const f32x4_t a = ld_nt<f32x4_t>(p), b = ld_nt<f32x4_t>(p + 4);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            f[j] = a[j];
            f[4 + j] = b[j];
        }
    } else if constexpr (V == 4) {
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
//
// Where the input current comes from is a policy:
//   DenseIn     -- x[T][N] in the I/O dtype (a layer fed by an ANN operator);
//   GainSpikeIn -- x[t][b][f] = gain[f] * spikes_in[t][b][f], read straight from the previous
//                  layer's spikes in any of the spike formats (a stack fused across its
//                  per-feature gain; the gain is rounded to the I/O dtype first, as a stored
//                  input current would be, and the backward multiplies by the same rounded
//                  gain, the exact derivative of that input current).
template <int IO, int V>
struct DenseIn {
    using raw = typename IoVec<IO, V>::raw;
    const void* x;
    __device__ raw load(int64_t N, int64_t t, int64_t n0) const { return IoVec<IO, V>::load(x, t * N + n0); }
    __device__ float get(const raw& r, int j, int64_t) const { return IoVec<IO, V>::get(r, j); }
};

template <int IO, int SPK, int V>
struct GainSpikeIn {
    // u8: V bytes; bits: the byte holding the lane's bits; io: V values of the I/O dtype
    using raw = std::conditional_t<SPK == SNN_SPK_IO, typename IoVec<IO, V>::raw,
                                   std::conditional_t<SPK == SNN_SPK_U8 && V == 8, uint64_t, uint32_t>>;
    const uint8_t* s;
    int64_t row_bytes;
    float gx[V];   // gain of the lane's neurons, rounded to the I/O dtype
    __device__ void init(const float* gain, int64_t F, int64_t n0, bool active) {
#pragma unroll
        for (int j = 0; j < V; ++j) gx[j] = io_round<IO>(active ? gain[(n0 + j) % F] : 0.0f);
    }
    __device__ raw load(int64_t N, int64_t t, int64_t n0) const {
        if constexpr (SPK == SNN_SPK_IO) {
            return IoVec<IO, V>::load(s, t * N + n0);
        } else {
            const uint8_t* row = s + t * row_bytes;
            if constexpr (SPK == SNN_SPK_BITS) return row[n0 >> 3];
            else if constexpr (V == 8) return *reinterpret_cast<const uint64_t*>(row + n0);
            else if constexpr (V == 4) return *reinterpret_cast<const uint32_t*>(row + n0);
            else if constexpr (V == 2) return *reinterpret_cast<const uint16_t*>(row + n0);
            else return row[n0];
        }
    }
    __device__ float get(const raw& r, int j, int64_t n0) const {
        if constexpr (SPK == SNN_SPK_IO) {
            return gx[j] * IoVec<IO, V>::get(r, j);   // spikes are 0 or 1: exact
        } else {
            const uint32_t bit =
                SPK == SNN_SPK_BITS ? uint32_t(r >> ((n0 + j) & 7)) & 1u : uint32_t(r >> (8 * j)) & 1u;
            return gx[j] * float(bit);
        }
    }
};

template <typename In, int K, bool FULL, bool REV>
__device__ __forceinline__ void load_rows(const In& in, typename In::raw (&buf)[K], int64_t N, int64_t t0, int kn,
                                          int64_t n0) {
    if constexpr (REV) {
#pragma unroll
        for (int i = K - 1; i >= 0; --i)
            if (FULL || i < kn) buf[i] = in.load(N, t0 + i, n0);
    } else {
#pragma unroll
        for (int i = 0; i < K; ++i)
            if (FULL || i < kn) buf[i] = in.load(N, t0 + i, n0);
    }
}

template <int IO, int SPK, int RESET, int V, int K, bool VOUT, bool FULL, bool ALL, typename In>
__device__ __forceinline__ void forward_rows(const LifK& c, const In& in, const typename In::raw (&xr)[K], int64_t N,
                                             int64_t t0, int kn, int64_t n0, bool active,
                                             uint8_t* __restrict__ spikes, int64_t row_bytes,
                                             float* __restrict__ v_out, float (&v)[V], bool (&y)[V]) {
    const bool on = ALL || active;
#pragma unroll
    for (int i = 0; i < K; ++i) {
        if (FULL || i < kn) {
#pragma unroll
            for (int j = 0; j < V; ++j) lif_step<RESET>(c, v[j], y[j], on ? in.get(xr[i], j, n0) : 0.0f);
            SpikeOut<IO, SPK, V>::store(spikes, row_bytes, t0 + i, n0, on, y);
            if (VOUT && on) store_f32<V>(v_out + (t0 + i) * N + n0, v);
        }
    }
}

// Forward of one workgroup's lanes.  Chunks 0 .. n_full-1 have K steps; a tail chunk of
// T % K steps follows when T % K != 0.  The membrane is checkpointed to saved[i][N] after
// step (i + 1) KC, for every such step before T: KC, the backward's chunk, is a multiple
// of K, since the forward may load a long chunk in shorter batches.  PIPE: double-buffered
// chunks -- the next chunk's rows are in flight while the current chunk is computed (for
// layers with few lanes, where occupancy alone cannot hide the memory latency); KC == K.
// Segment state (a sequence split along time): v_in, if not null, is the membrane the
// previous segment ended with, and the spike state entering the first step is v_in >= V_th;
// v_last, if not null, receives the membrane after the last step.
template <int IO, int SPK, int RESET, int V, int K, int KC, bool VOUT, bool PIPE, bool ALL, typename In,
          bool SYNC = false>
__device__ __forceinline__ void forward_lanes(const LifK& c, const In& in, int64_t T, int64_t N, int64_t n0,
                                              uint8_t* __restrict__ spikes, int64_t row_bytes,
                                              float* __restrict__ saved, float* __restrict__ v_out,
                                              const float* __restrict__ v_in, float* __restrict__ v_last) {
    using raw = typename In::raw;
    const bool active = ALL || n0 < N;
    float v[V];
    bool y[V];
#pragma unroll
    for (int j = 0; j < V; ++j) {
        v[j] = c.rest;  // v^0 = V_rest
        y[j] = false;   // no spike before the first step
    }
    if (v_in != nullptr && (ALL || active)) {
        load_f32<V>(v_in + n0, v);
#pragma unroll
        for (int j = 0; j < V; ++j) y[j] = v[j] >= c.th;
    }
    const int64_t n_full = T / K;
    const int k_tail = int(T % K);
    const int64_t last = k_tail ? n_full : n_full - 1;   // index of the last chunk
    // The scheduler must not move a chunk's compute across the batch of loads that
    // precedes it: that would change the outstanding-operation count between loop entry
    // and back-edge and make the compiler's waits conservative.
    auto load = [&](raw (&buf)[K], int64_t ch) {
        __builtin_amdgcn_sched_barrier(0);
        if (ALL || active) load_rows<In, K, true, false>(in, buf, N, ch * K, K, n0);
        __builtin_amdgcn_sched_barrier(0);
    };
    static_assert(KC % K == 0 && (!PIPE || KC == K), "checkpoint interval");
    // ckpt: true_type = this chunk is never the last (checkpoint unconditionally)
    auto step = [&](const raw (&buf)[K], int64_t ch, auto ckpt) {
        forward_rows<IO, SPK, RESET, V, K, VOUT, true, ALL>(c, in, buf, N, ch * K, K, n0, active, spikes, row_bytes,
                                                            v_out, v, y);
        if constexpr (KC == K) {
            if ((decltype(ckpt)::value || ch < last) && (ALL || active)) store_f32<V>(saved + ch * N + n0, v);
        } else {
            const int64_t t_end = (ch + 1) * K;
            if (t_end % KC == 0 && t_end < T && (ALL || active)) store_f32<V>(saved + (t_end / KC - 1) * N + n0, v);
        }
    };
    constexpr std::true_type not_last{};
    constexpr std::false_type maybe_last{};
    raw a[K];
    if constexpr (!PIPE) {
        for (int64_t ch = 0; ch < n_full; ++ch) {
            load(a, ch);
            step(a, ch, maybe_last);
            if constexpr (SYNC) __syncthreads();   // the workgroup's waves walk the rows in step
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
        if (ALL || active) load_rows<In, K, false, false>(in, a, N, n_full * K, k_tail, n0);
        forward_rows<IO, SPK, RESET, V, K, VOUT, false, ALL>(c, in, a, N, n_full * K, k_tail, n0, active, spikes,
                                                             row_bytes, v_out, v, y);
    }
    if (v_last != nullptr && (ALL || active)) store_f32<V>(v_last + n0, v);
}

// Grid: one lane per V neurons over ceil(max(N, 8*row_bytes) / V) lanes.  Lanes at or beyond
// N load nothing and report no spikes; they exist only to complete spike-bit words.
// BLK: the workgroup size; above kBlock (layers of several chunks, not double-buffered)
// the waves of a workgroup that lies wholly inside N meet at a barrier after every chunk.
template <int IO, int SPK, int RESET, int V, int K, int KC, bool VOUT, bool PIPE, int BLK = kBlock>
__global__ __launch_bounds__(BLK) void lif_forward_kernel(LifK c, int64_t T, int64_t N,
                                                          const void* __restrict__ x,
                                                          uint8_t* __restrict__ spikes,
                                                          int64_t row_bytes,
                                                          float* __restrict__ saved,
                                                          float* __restrict__ v_out,
                                                          const float* __restrict__ v_in,
                                                          float* __restrict__ v_last) {
    static_assert(BLK == kBlock || !PIPE, "barriers only in the single-buffered chunk loop");
    const int64_t first = xcd_contiguous_block() * BLK * V;
    const int64_t n0 = first + int64_t(threadIdx.x) * V;
    const DenseIn<IO, V> in{x};
    if (first + BLK * V <= N)
        forward_lanes<IO, SPK, RESET, V, K, KC, VOUT, PIPE, true, DenseIn<IO, V>, (BLK > kBlock)>(
            c, in, T, N, n0, spikes, row_bytes, saved, v_out, v_in, v_last);
    else
        forward_lanes<IO, SPK, RESET, V, K, KC, VOUT, PIPE, false>(c, in, T, N, n0, spikes, row_bytes, saved, v_out,
                                                               v_in, v_last);
}

// The same forward with the input current read from the previous layer's spikes through
// the per-feature gain (neuron n has feature n % F).  Spikes in and out share the format.
// Its chunks are single-buffered: a spike word per lane and row is too little to hide
// behind a second buffer's registers.
template <int IO, int SPK, int RESET, int V, int K, int KC, bool VOUT>
__global__ __launch_bounds__(kBlock) void lif_forward_gain_kernel(LifK c, int64_t T, int64_t N, int64_t F,
                                                                  const uint8_t* __restrict__ spikes_in,
                                                                  const float* __restrict__ gain,
                                                                  uint8_t* __restrict__ spikes,
                                                                  int64_t row_bytes,
                                                                  float* __restrict__ saved,
                                                                  float* __restrict__ v_out) {
    const int64_t first = xcd_contiguous_block() * kBlock * V;
    const int64_t n0 = first + int64_t(threadIdx.x) * V;
    GainSpikeIn<IO, SPK, V> in;
    in.s = spikes_in;
    in.row_bytes = row_bytes;
    in.init(gain, F, n0, n0 < N);
    if (first + kBlock * V <= N)
        forward_lanes<IO, SPK, RESET, V, K, KC, VOUT, false, true>(c, in, T, N, n0, spikes, row_bytes, saved, v_out,
                                                              nullptr, nullptr);
    else
        forward_lanes<IO, SPK, RESET, V, K, KC, VOUT, false, false>(c, in, T, N, n0, spikes, row_bytes, saved, v_out,
                                                               nullptr, nullptr);
}

// Backward of one chunk.  v/y enter as the state before the chunk's first step; g enters
// as dL/dv of the step after the chunk and leaves as dL/dv of the chunk's first step.
// GAIN: the stored gradient is the fused stack's dL/dy of the previous layer,
// gain[f] * dL/dx, instead of dL/dx.
template <int IO, int RESET, int V, int K, bool FULL, bool GAIN, typename In>
__device__ __forceinline__ void backward_rows(const LifK& c, const In& in, const typename In::raw (&xr)[K],
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
                lif_step<RESET>(c, v[j], y[j], in.get(xr[i], j, n0));
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
                if constexpr (GAIN) out[j] = in.gx[j] * g[j];
                else out[j] = g[j];
            }
            Io::store(gx, (t0 + i) * N + n0, out);
        }
    }
}

// Everything the backward of chunk ch reads: the state entering it (loaded first), its
// input rows, and its dL/dy rows (issued last-first, the order the reverse pass uses them).
template <int IO, int V, int K, typename In>
struct BwdChunk {
    typename In::raw x[K];
    typename IoVec<IO, V>::raw gs[K];
    float v[V];
};

// Segment state of the backward (a sequence split along time): v_in as in the forward;
// g_in, if not null, is dL/dv^{T+1}, the gradient the following segment hands back (else
// 0); g_out, if not null, receives dL/dv^1 in fp32 for the preceding segment.
struct BwdSeg {
    const float* v_in;
    const float* g_in;
    float* g_out;
};

// ALWAYS: the layer has a checkpoint row, so the state is loaded unconditionally (chunk 0
// reads v_in, or row 0 and then takes V_rest instead), keeping the caller's loop free of
// branches.
template <int IO, int V, int K, bool FULL, bool ALWAYS, typename In>
__device__ __forceinline__ void backward_load(BwdChunk<IO, V, K, In>& b, const LifK& c, const In& in,
                                              const float* __restrict__ saved, const float* v_in, const void* gs,
                                              int64_t N, int64_t ch, int kn, int64_t n0) {
    if (ALWAYS) {
        load_f32<V>((ch > 0 ? saved + (ch - 1) * N : v_in != nullptr ? v_in : saved) + n0, b.v);
    } else if (ch > 0) {
        load_f32<V>(saved + (ch - 1) * N + n0, b.v);
    } else if (v_in != nullptr) {
        load_f32<V>(v_in + n0, b.v);
    } else {
#pragma unroll
        for (int j = 0; j < V; ++j) b.v[j] = c.rest;
    }
    load_rows<In, K, FULL, false>(in, b.x, N, ch * K, kn, n0);
    load_rows<DenseIn<IO, V>, K, FULL, true>(DenseIn<IO, V>{gs}, b.gs, N, ch * K, kn, n0);
}

template <int IO, int RESET, int V, int K, bool FULL, bool GAIN, typename In>
__device__ __forceinline__ void backward_chunk(const LifK& c, const In& in, const BwdChunk<IO, V, K, In>& b,
                                               bool has_v_in, int64_t N, int64_t ch, int kn, int64_t n0, void* gx,
                                               float (&g)[V]) {
    // a checkpoint (or v_in) is a post-step membrane with spike state v >= V_th; the
    // sequence itself starts at V_rest with no spike
    const bool carried = ch > 0 || has_v_in;
    float v[V];
    bool y[V];
#pragma unroll
    for (int j = 0; j < V; ++j) {
        v[j] = carried ? b.v[j] : c.rest;
        y[j] = carried && b.v[j] >= c.th;
    }
    backward_rows<IO, RESET, V, K, FULL, GAIN>(c, in, b.x, b.gs, N, ch * K, kn, n0, gx, v, y, g);
}

// Chunks are processed last-first: the short tail chunk (if any), then the full chunks.
template <int IO, int RESET, int V, int K, bool PIPE, bool GAIN, typename In, bool SYNC = false>
__device__ __forceinline__ void backward_lanes(const LifK& c, const In& in, int64_t T, int64_t N, int64_t n0,
                                               const float* __restrict__ saved, const void* gs, void* gx,
                                               const BwdSeg& seg) {
    using Chunk = BwdChunk<IO, V, K, In>;
    float g[V];
    if (seg.g_in != nullptr) {
        load_f32<V>(seg.g_in + n0, g);
    } else {
#pragma unroll
        for (int j = 0; j < V; ++j) g[j] = 0.0f;  // dL/dv^{T+1} = 0
    }
    const bool has_v_in = seg.v_in != nullptr;
    const int64_t n_full = T / K;
    const int k_tail = int(T % K);
    Chunk a;
    if (k_tail) {
        backward_load<IO, V, K, false, false>(a, c, in, saved, seg.v_in, gs, N, n_full, k_tail, n0);
        backward_chunk<IO, RESET, V, K, false, GAIN>(c, in, a, has_v_in, N, n_full, k_tail, n0, gx, g);
    }
    auto load = [&](Chunk& buf, int64_t ch) {
        __builtin_amdgcn_sched_barrier(0);
        backward_load<IO, V, K, true, PIPE>(buf, c, in, saved, seg.v_in, gs, N, ch, K, n0);
        __builtin_amdgcn_sched_barrier(0);
    };
    auto step = [&](const Chunk& buf, int64_t ch) {
        backward_chunk<IO, RESET, V, K, true, GAIN>(c, in, buf, has_v_in, N, ch, K, n0, gx, g);
    };
    if constexpr (!PIPE) {
        for (int64_t ch = n_full - 1; ch >= 0; --ch) {
            load(a, ch);
            step(a, ch);
            if constexpr (SYNC) __syncthreads();   // the workgroup's waves walk the rows in step
        }
    } else if (n_full > 0) {
        Chunk b;
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
    if (seg.g_out != nullptr) store_f32<V>(seg.g_out + n0, g);
}

// BLK: the workgroup size.  SYNC: its waves meet at a barrier after every chunk (only in
// a workgroup wholly inside N; one that is not drops its lanes beyond N).
template <int IO, int RESET, int V, int K, bool PIPE, int BLK = kBlock, bool SYNC = false>
__global__ __launch_bounds__(BLK) void lif_backward_kernel(LifK c, int64_t T, int64_t N,
                                                           const void* __restrict__ x,
                                                           const float* __restrict__ saved,
                                                           const void* gs, void* gx, BwdSeg seg) {
    static_assert(!SYNC || !PIPE, "barriers only in the single-buffered chunk loop");
    const int64_t first = xcd_contiguous_block() * BLK * V;
    const int64_t n0 = first + int64_t(threadIdx.x) * V;
    const DenseIn<IO, V> in{x};
    if (first + BLK * V <= N) {
        backward_lanes<IO, RESET, V, K, PIPE, false, DenseIn<IO, V>, SYNC>(c, in, T, N, n0, saved, gs, gx, seg);
        return;
    }
    if (n0 >= N) return;
    backward_lanes<IO, RESET, V, K, PIPE, false>(c, in, T, N, n0, saved, gs, gx, seg);
}

// Backward of the gain-fed layer: recomputes from the previous layer's spikes and writes
// gain[f] * dL/dx, the gradient with respect to those spikes (single-buffered chunks).
template <int IO, int SPK, int RESET, int V, int K>
__global__ __launch_bounds__(kBlock) void lif_backward_gain_kernel(LifK c, int64_t T, int64_t N, int64_t F,
                                                                   const uint8_t* __restrict__ spikes_in,
                                                                   const float* __restrict__ gain,
                                                                   int64_t row_bytes,
                                                                   const float* __restrict__ saved,
                                                                   const void* gs, void* gs_in) {
    const int64_t first = xcd_contiguous_block() * kBlock * V;
    const int64_t n0 = first + int64_t(threadIdx.x) * V;
    if (first + kBlock * V > N && n0 >= N) return;
    GainSpikeIn<IO, SPK, V> in;
    in.s = spikes_in;
    in.row_bytes = row_bytes;
    in.init(gain, F, n0, true);
    backward_lanes<IO, RESET, V, K, false, true>(c, in, T, N, n0, saved, gs, gs_in, BwdSeg{nullptr, nullptr, nullptr});
}

// ------------------------------------------------------------------------------------
// A stack of L layers fused across depth as well as time.  Layer 0 is fed x; layer l > 0 is
// fed gain_{l-1}[f] y_{l-1} of the same step (neuron n has feature n % F), so one lane can
// carry its neurons through every layer with all L membranes in VGPRs.  Only x, the last
// layer's spikes, the checkpoints (all L membranes every K steps, saved[chunk][l][N]) and,
// backward, the last layer's dL/dy and layer 0's dL/dx go through memory.  The gain is
// rounded to the I/O dtype before it multiplies a spike, as a stored input current would
// be, and the gradient handed down a layer is that rounded gain times dL/dx, kept in fp32.
template <int V, int L>
struct StackGains {
    float gx[L - 1][V];   // rounded to the I/O dtype
    template <int IO>
    __device__ void init(const float* gains, int64_t F, int64_t n0, bool active) {
#pragma unroll
        for (int l = 0; l < L - 1; ++l) {
#pragma unroll
            for (int j = 0; j < V; ++j) gx[l][j] = io_round<IO>(active ? gains[l * F + (n0 + j) % F] : 0.0f);
        }
    }
};

// One step of every layer; x0 is layer 0's input current.
template <int RESET, int V, int L>
__device__ __forceinline__ void stack_step(const LifK& c, const StackGains<V, L>& G, const float (&x0)[V],
                                           float (&v)[L][V], bool (&y)[L][V]) {
#pragma unroll
    for (int j = 0; j < V; ++j) lif_step<RESET>(c, v[0][j], y[0][j], x0[j]);
#pragma unroll
    for (int l = 1; l < L; ++l) {
#pragma unroll
        for (int j = 0; j < V; ++j) lif_step<RESET>(c, v[l][j], y[l][j], G.gx[l - 1][j] * float(y[l - 1][j]));
    }
}

// Forward of one workgroup's lanes, chunks of K steps (a short tail chunk last).  OUT: also
// write the hidden layers' spikes (hidden[l][T][row_bytes]) and every layer's membrane
// (v_out[l][T][N]) where those pointers are not null.
template <int IO, int SPK, int RESET, int V, int K, int L, bool OUT, bool ALL>
__device__ __forceinline__ void stack_forward_lanes(const LifK& c, const DenseIn<IO, V>& in,
                                                    const StackGains<V, L>& G, int64_t T, int64_t N, int64_t n0,
                                                    uint8_t* __restrict__ spikes, uint8_t* __restrict__ hidden,
                                                    int64_t row_bytes, float* __restrict__ saved,
                                                    float* __restrict__ v_out) {
    using raw = typename DenseIn<IO, V>::raw;
    const bool active = ALL || n0 < N;
    float v[L][V];
    bool y[L][V];
#pragma unroll
    for (int l = 0; l < L; ++l) {
#pragma unroll
        for (int j = 0; j < V; ++j) {
            v[l][j] = c.rest;
            y[l][j] = false;
        }
    }
    const int64_t n_full = T / K;
    const int k_tail = int(T % K);
    const int64_t last = k_tail ? n_full : n_full - 1;
    raw a[K];
    auto rows = [&](int64_t t0, int kn, auto full) {
#pragma unroll
        for (int i = 0; i < K; ++i) {
            if (decltype(full)::value || i < kn) {
                float x0[V];
#pragma unroll
                for (int j = 0; j < V; ++j) x0[j] = active ? in.get(a[i], j, n0) : 0.0f;
                stack_step<RESET, V, L>(c, G, x0, v, y);
                const int64_t t = t0 + i;
                SpikeOut<IO, SPK, V>::store(spikes, row_bytes, t, n0, active, y[L - 1]);
                if constexpr (OUT) {
                    if (hidden != nullptr) {
#pragma unroll
                        for (int l = 0; l < L - 1; ++l)
                            SpikeOut<IO, SPK, V>::store(hidden + l * T * row_bytes, row_bytes, t, n0, active, y[l]);
                    }
                    if (v_out != nullptr && active) {
#pragma unroll
                        for (int l = 0; l < L; ++l) store_f32<V>(v_out + (l * T + t) * N + n0, v[l]);
                    }
                }
            }
        }
    };
    for (int64_t ch = 0; ch < n_full; ++ch) {
        __builtin_amdgcn_sched_barrier(0);
        if (active) load_rows<DenseIn<IO, V>, K, true, false>(in, a, N, ch * K, K, n0);
        __builtin_amdgcn_sched_barrier(0);
        rows(ch * K, K, std::true_type{});
        if (ch < last && active) {
#pragma unroll
            for (int l = 0; l < L; ++l) store_f32<V>(saved + (ch * L + l) * N + n0, v[l]);
        }
    }
    if (k_tail) {
        if (active) load_rows<DenseIn<IO, V>, K, false, false>(in, a, N, n_full * K, k_tail, n0);
        rows(n_full * K, k_tail, std::false_type{});
    }
}

// Grid: one lane per V neurons over ceil(max(N, 8*row_bytes) / V) lanes (as the layer's
// forward); gains is [L-1][F].
template <int IO, int SPK, int RESET, int V, int K, int L, bool OUT>
__global__ __launch_bounds__(kBlock) void lif_stack_forward_kernel(LifK c, int64_t T, int64_t N, int64_t F,
                                                                   const void* __restrict__ x,
                                                                   const float* __restrict__ gains,
                                                                   uint8_t* __restrict__ spikes,
                                                                   uint8_t* __restrict__ hidden,
                                                                   int64_t row_bytes,
                                                                   float* __restrict__ saved,
                                                                   float* __restrict__ v_out) {
    const int64_t first = xcd_contiguous_block() * kBlock * V;
    const int64_t n0 = first + int64_t(threadIdx.x) * V;
    const DenseIn<IO, V> in{x};
    StackGains<V, L> G;
    G.template init<IO>(gains, F, n0, n0 < N);
    if (first + kBlock * V <= N)
        stack_forward_lanes<IO, SPK, RESET, V, K, L, OUT, true>(c, in, G, T, N, n0, spikes, hidden, row_bytes, saved,
                                                                v_out);
    else
        stack_forward_lanes<IO, SPK, RESET, V, K, L, OUT, false>(c, in, G, T, N, n0, spikes, hidden, row_bytes,
                                                                 saved, v_out);
}

// Backward of one chunk: recompute every layer's membranes from the state entering the
// chunk (checkpoint or V_rest), then Eq. (3) in reverse time, the layers top-down within
// each step: the gradient layer l hands down, gain_{l-1} g_l, is layer l-1's dL/dy of the
// same step.  g[l] enters as dL/dv of layer l at the step after the chunk.
template <int IO, int RESET, int V, int K, int L, bool FULL>
__device__ __forceinline__ void stack_backward_chunk(const LifK& c, const DenseIn<IO, V>& in,
                                                     const StackGains<V, L>& G,
                                                     const typename IoVec<IO, V>::raw (&xr)[K],
                                                     const typename IoVec<IO, V>::raw (&gr)[K],
                                                     const float (&vc)[L][V], bool carried, int64_t N, int64_t t0,
                                                     int kn, int64_t n0, void* gx, float (&g)[L][V]) {
    using Io = IoVec<IO, V>;
    float v[L][V];
    bool y[L][V];
#pragma unroll
    for (int l = 0; l < L; ++l) {
#pragma unroll
        for (int j = 0; j < V; ++j) {
            v[l][j] = carried ? vc[l][j] : c.rest;
            y[l][j] = carried && vc[l][j] >= c.th;
        }
    }
    float vs[K][L][V];
#pragma unroll
    for (int i = 0; i < K; ++i) {
        if (FULL || i < kn) {
            float x0[V];
#pragma unroll
            for (int j = 0; j < V; ++j) x0[j] = in.get(xr[i], j, n0);
            stack_step<RESET, V, L>(c, G, x0, v, y);
#pragma unroll
            for (int l = 0; l < L; ++l) {
#pragma unroll
                for (int j = 0; j < V; ++j) vs[i][l][j] = v[l][j];
            }
        }
    }
#pragma unroll
    for (int i = K - 1; i >= 0; --i) {
        if (FULL || i < kn) {
            float out[V];
#pragma unroll
            for (int j = 0; j < V; ++j) {
                float gs = Io::get(gr[i], j);
#pragma unroll
                for (int l = L - 1; l >= 0; --l) {
                    const float vt = vs[i][l][j];
                    const float d = surrogate(c, vt - c.th);
                    float dv_next;
                    if (RESET == SNN_RESET_HARD)  // k (1 - y^t) + (V_rest - k v^t) delta^t
                        dv_next = fmaf(fmaf(-c.k, vt, c.rest), d, vt >= c.th ? 0.0f : c.k);
                    else                          // k (1 - V_th delta^t)
                        dv_next = fmaf(-c.kth, d, c.k);
                    g[l][j] = fmaf(gs, d, dv_next * g[l][j]);
                    if (l > 0) gs = G.gx[l - 1][j] * g[l][j];
                }
                out[j] = g[0][j];
            }
            Io::store(gx, (t0 + i) * N + n0, out);
        }
    }
}

template <int IO, int RESET, int V, int K, int L>
__device__ __forceinline__ void stack_backward_lanes(const LifK& c, const DenseIn<IO, V>& in,
                                                     const StackGains<V, L>& G, int64_t T, int64_t N, int64_t n0,
                                                     const float* __restrict__ saved, const void* gs, void* gx) {
    using raw = typename IoVec<IO, V>::raw;
    float g[L][V];
#pragma unroll
    for (int l = 0; l < L; ++l) {
#pragma unroll
        for (int j = 0; j < V; ++j) g[l][j] = 0.0f;   // dL/dv^{T+1} = 0 in every layer
    }
    const int64_t n_full = T / K;
    const int k_tail = int(T % K);
    raw xr[K], gr[K];
    float vc[L][V];
    auto load = [&](int64_t ch, int kn, auto full) {
        if (ch > 0) {
#pragma unroll
            for (int l = 0; l < L; ++l) load_f32<V>(saved + ((ch - 1) * L + l) * N + n0, vc[l]);
        }
        load_rows<DenseIn<IO, V>, K, decltype(full)::value, false>(in, xr, N, ch * K, kn, n0);
        load_rows<DenseIn<IO, V>, K, decltype(full)::value, true>(DenseIn<IO, V>{gs}, gr, N, ch * K, kn, n0);
    };
    if (k_tail) {
        load(n_full, k_tail, std::false_type{});
        stack_backward_chunk<IO, RESET, V, K, L, false>(c, in, G, xr, gr, vc, n_full > 0, N, n_full * K, k_tail, n0,
                                                        gx, g);
    }
    for (int64_t ch = n_full - 1; ch >= 0; --ch) {
        __builtin_amdgcn_sched_barrier(0);
        load(ch, K, std::true_type{});
        __builtin_amdgcn_sched_barrier(0);
        stack_backward_chunk<IO, RESET, V, K, L, true>(c, in, G, xr, gr, vc, ch > 0, N, ch * K, K, n0, gx, g);
    }
}

template <int IO, int RESET, int V, int K, int L>
__global__ __launch_bounds__(kBlock) void lif_stack_backward_kernel(LifK c, int64_t T, int64_t N, int64_t F,
                                                                    const void* __restrict__ x,
                                                                    const float* __restrict__ gains,
                                                                    const float* __restrict__ saved,
                                                                    const void* gs, void* gx) {
    const int64_t first = xcd_contiguous_block() * kBlock * V;
    const int64_t n0 = first + int64_t(threadIdx.x) * V;
    if (first + kBlock * V > N && n0 >= N) return;
    StackGains<V, L> G;
    G.template init<IO>(gains, F, n0, true);
    stack_backward_lanes<IO, RESET, V, K, L>(c, DenseIn<IO, V>{x}, G, T, N, n0, saved, gs, gx);
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
    if constexpr (SPK == SNN_SPK_IO) {   // spikes already 0/1 in the I/O dtype
        using Io = IoVec<IO, V>;
        auto emit = [&](const typename Io::raw& r, int64_t t) {
            float out[V];
#pragma unroll
            for (int j = 0; j < V; ++j) out[j] = gv[j] * Io::get(r, j);
            Io::store(x_next, t * N + n0, out);
        };
        int64_t t0 = 0;
        for (; t0 + kGlueRows <= T; t0 += kGlueRows) {
            typename Io::raw r[kGlueRows];
#pragma unroll
            for (int i = 0; i < kGlueRows; ++i) r[i] = Io::load(spikes, (t0 + i) * N + n0);
#pragma unroll
            for (int i = 0; i < kGlueRows; ++i) emit(r[i], t0 + i);
        }
        for (; t0 < T; ++t0) emit(Io::load(spikes, t0 * N + n0), t0);
    } else {
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
}

template <int IO, int V>
__global__ __launch_bounds__(kBlock) void gain_backward_kernel(int64_t T, int64_t N, int64_t F,
                                                               const void* gx_next,
                                                               const float* __restrict__ gain,
                                                               void* gs) {
    using Io = IoVec<IO, V>;
    const int64_t n0 = (xcd_contiguous_block() * kBlock + threadIdx.x) * V;
    if (n0 >= N) return;
    float gv[V];   // the gain as the forward applies it (rounded to the I/O dtype)
#pragma unroll
    for (int j = 0; j < V; ++j) gv[j] = io_round<IO>(gain[(n0 + j) % F]);
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
// The same gain over a flat layout.  When every row is whole (N a multiple of the piece
// width W, spike rows without padding) the [T][N] tensors are one contiguous run of T*N
// elements and the gain is elementwise: element e belongs to feature e % F, N being a
// multiple of F.  Lanes then stream consecutive 16-byte pieces of the whole run, the
// access pattern of a plain copy, instead of walking rows N elements apart.  F is a
// multiple of W, so a piece never wraps around the features and its W gains are one
// aligned vector load; a lane loads the gains of all its pieces before their data, so
// that the in-order wait counter never holds a piece's arithmetic behind a later load.
constexpr int kFlatPieces = 8;   // pieces per lane, all loads in flight together

template <int IO>
constexpr int flat_width() { return IO == SNN_IO_F32 ? 4 : 8; }   // elements per 16-byte output piece

template <int W>
struct FlatGains {
    float g[W];
    __device__ void load(const float* gain, int64_t f) {
#pragma unroll
        for (int h = 0; h < W / 4; ++h) {
            const f32x4_t v = *reinterpret_cast<const f32x4_t*>(gain + f + 4 * h);
#pragma unroll
            for (int j = 0; j < 4; ++j) g[4 * h + j] = v[j];
        }
    }
};

// The spikes of one piece (W consecutive elements from element e) as one raw word.
template <int IO, int SPK>
struct FlatSpikes {   // SNN_SPK_IO: 0/1 in the I/O dtype
    using Io = IoVec<IO, flat_width<IO>()>;
    using raw = typename Io::raw;
    __device__ static raw load(const uint8_t* s, int64_t e) { return Io::load(s, e); }
    __device__ static float get(const raw& r, int j) { return Io::get(r, j); }
};

template <int IO>
struct FlatSpikes<IO, SNN_SPK_U8> {
    static constexpr int W = flat_width<IO>();
    using raw = std::conditional_t<W == 4, uint32_t, uint64_t>;
    __device__ static raw load(const uint8_t* s, int64_t e) { return *reinterpret_cast<const raw*>(s + e); }
    __device__ static float get(const raw& r, int j) { return float(uint32_t(r >> (8 * j)) & 0xffu); }
};

template <int IO>
struct FlatSpikes<IO, SNN_SPK_BITS> {   // W bits of byte e / 8, from bit e % 8 (0, or 4 when W = 4)
    using raw = uint32_t;
    __device__ static raw load(const uint8_t* s, int64_t e) { return uint32_t(s[e >> 3]) >> (e & 7); }
    __device__ static float get(const raw& r, int j) { return float((r >> j) & 1u); }
};

// Runs emit(raw, gains, e) over the lane's pieces, e the piece's first element.  A lane's
// pieces are kBlock pieces apart, so a wave touches one contiguous kilobyte per piece and
// a workgroup one contiguous run.  Workgroups take the runs in launch order, i.e. dealt
// round-robin over the XCDs: for this flat stream that measured faster than giving each
// XCD one contiguous range, as the row walks do (stack workload, gain backward 26.6 vs
// 28.4 us).  `step` = kBlock * W % F, precomputed by the host.
template <int W, typename Raw, typename Load, typename Emit>
__device__ __forceinline__ void flat_pieces(int64_t pieces, int64_t F, int64_t step, const float* gain, Load load,
                                            Emit emit) {
    const int64_t base = int64_t(blockIdx.x) * (kBlock * kFlatPieces);
    const int64_t p0 = base + threadIdx.x;
    int64_t f = (p0 * W) % F;
    FlatGains<W> g[kFlatPieces];
    Raw r[kFlatPieces];
    if (base + kBlock * kFlatPieces <= pieces) {   // the whole workgroup inside: no per-lane guards
#pragma unroll
        for (int u = 0; u < kFlatPieces; ++u) {
            g[u].load(gain, f);
            f += step;
            if (f >= F) f -= F;
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < kFlatPieces; ++u) r[u] = load((p0 + u * kBlock) * W);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < kFlatPieces; ++u) emit(r[u], g[u], (p0 + u * kBlock) * W);
    } else {
#pragma unroll
        for (int u = 0; u < kFlatPieces; ++u) {
            const int64_t p = p0 + u * kBlock;
            if (p < pieces) {
                g[u].load(gain, f);
                emit(load(p * W), g[u], p * W);
            }
            f += step;
            if (f >= F) f -= F;
        }
    }
}

template <int IO, int SPK>
__global__ __launch_bounds__(kBlock) void gain_forward_flat_kernel(int64_t pieces, int64_t F, int64_t step,
                                                                   const uint8_t* __restrict__ spikes,
                                                                   const float* __restrict__ gain,
                                                                   void* __restrict__ x_next) {
    constexpr int W = flat_width<IO>();
    using In = FlatSpikes<IO, SPK>;
    flat_pieces<W, typename In::raw>(
        pieces, F, step, gain, [&](int64_t e) { return In::load(spikes, e); },
        [&](const typename In::raw& r, const FlatGains<W>& g, int64_t e) {
            float out[W];
#pragma unroll
            for (int j = 0; j < W; ++j) out[j] = g.g[j] * In::get(r, j);
            IoVec<IO, W>::store(x_next, e, out);
        });
}

// gx_next and gs may be the same buffer: every element is read and written by one lane,
// its load first.
template <int IO>
__global__ __launch_bounds__(kBlock) void gain_backward_flat_kernel(int64_t pieces, int64_t F, int64_t step,
                                                                    const void* gx_next,
                                                                    const float* __restrict__ gain, void* gs) {
    constexpr int W = flat_width<IO>();
    using Io = IoVec<IO, W>;
    flat_pieces<W, typename Io::raw>(
        pieces, F, step, gain, [&](int64_t e) { return Io::load(gx_next, e); },
        [&](const typename Io::raw& r, const FlatGains<W>& g, int64_t e) {
            float out[W];   // the gain as the forward applies it (rounded to the I/O dtype)
#pragma unroll
            for (int j = 0; j < W; ++j) out[j] = io_round<IO>(g.g[j]) * Io::get(r, j);
            Io::store(gs, e, out);
        });
}

}  // namespace snnlif

namespace snnlif {

// ------------------------------------------------------------------------------------
// Serial (per-time-step) baseline: the method temporal fusion replaces (Fig. 3).  One
// launch per step; the membrane state round-trips through memory between steps.  The
// arithmetic is the fused kernels' own (lif_step, surrogate, the Eq. (3) update), so the
// results are identical bit for bit.

// Step t: v_prev (fp32, NULL before the first step: V_rest, no spike) -> v_t, spikes_t.
template <int IO, int SPK, int RESET, int V>
__global__ __launch_bounds__(kBlock) void lif_serial_forward_kernel(LifK c, int64_t N, const void* __restrict__ x_t,
                                                                    const float* __restrict__ v_prev,
                                                                    float* __restrict__ v_t,
                                                                    uint8_t* __restrict__ spikes_t,
                                                                    int64_t row_bytes) {
    using Io = IoVec<IO, V>;
    const int64_t n0 = (int64_t(blockIdx.x) * kBlock + threadIdx.x) * V;
    const bool active = n0 < N;
    float v[V];
    bool y[V];
    typename Io::raw xr;
    if (active) {
        xr = Io::load(x_t, n0);
        if (v_prev != nullptr) load_f32<V>(v_prev + n0, v);
    }
#pragma unroll
    for (int j = 0; j < V; ++j) {
        if (v_prev == nullptr || !active) v[j] = c.rest;
        y[j] = v_prev != nullptr && active && v[j] >= c.th;
        lif_step<RESET>(c, v[j], y[j], active ? Io::get(xr, j) : 0.0f);
    }
    SpikeOut<IO, SPK, V>::store(spikes_t, row_bytes, 0, n0, active, y);
    if (active) store_f32<V>(v_t + n0, v);
}

// Step t, reverse time: v_t, dL/dy_t, g_next = dL/dv_{t+1} (fp32, NULL at the last step)
// -> dL/dx_t (I/O dtype) and, if g_out is not NULL, dL/dv_t in fp32 for the next call.
template <int IO, int RESET, int V>
__global__ __launch_bounds__(kBlock) void lif_serial_backward_kernel(LifK c, int64_t N, const float* __restrict__ v_t,
                                                                     const void* gs_t, const float* g_next,
                                                                     void* gx_t, float* g_out) {
    using Io = IoVec<IO, V>;
    const int64_t n0 = (int64_t(blockIdx.x) * kBlock + threadIdx.x) * V;
    if (n0 >= N) return;
    float vt[V], g[V], out[V];
    load_f32<V>(v_t + n0, vt);
    if (g_next != nullptr) load_f32<V>(g_next + n0, g);
    const typename Io::raw gr = Io::load(gs_t, n0);
#pragma unroll
    for (int j = 0; j < V; ++j) {
        if (g_next == nullptr) g[j] = 0.0f;
        const float d = surrogate(c, vt[j] - c.th);
        float dv_next;
        if (RESET == SNN_RESET_HARD)
            dv_next = fmaf(fmaf(-c.k, vt[j], c.rest), d, vt[j] >= c.th ? 0.0f : c.k);
        else
            dv_next = fmaf(-c.kth, d, c.k);
        out[j] = fmaf(Io::get(gr, j), d, dv_next * g[j]);
    }
    Io::store(gx_t, n0, out);
    if (g_out != nullptr) store_f32<V>(g_out + n0, out);
}

}  // namespace snnlif
