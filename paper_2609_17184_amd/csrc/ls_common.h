// Device-side definitions shared by the LoopSpec gfx950 kernels and the host
// runtime that launches them.
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ls {

// Kernel timing for the decode profiler: when armed, the next launch made
// through ls_launch carries the two events in its own dispatch, so they take
// the kernel's start and end times (what a kernel trace reports), not the
// stream's progress around the launch.
struct LaunchProbe {
    hipEvent_t start = nullptr, stop = nullptr;
    bool armed = false;
};
inline LaunchProbe& launch_probe() {
    static thread_local LaunchProbe p;
    return p;
}
inline hipError_t ls_launch(const void* f, dim3 grid, dim3 block, void** args, size_t lds, hipStream_t st) {
    LaunchProbe& pr = launch_probe();
    if (pr.armed) {
        pr.armed = false;
        return hipExtLaunchKernel(f, grid, block, args, lds, st, pr.start, pr.stop, 0);
    }
    return hipLaunchKernel(f, grid, block, args, lds, st);
}

// ---------------------------------------------------------------------------
// small vector types
// ---------------------------------------------------------------------------
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

constexpr int kTile = 16;            // output features per MFMA tile (and per sum-of-squares partial)
constexpr int kMaxRows = 64;         // rows (branches) one batched pass handles
constexpr int kChunk = 64;           // attention positions per split-softmax chunk
constexpr int kChainMax = 24;        // in-flight ancestors a row can have (positions tdone .. pos-1)

// Thread index as a value the compiler cannot hoist: per-phase geometry is
// then recomputed where it is used instead of being held in registers across
// the phases of a persistent kernel.
// Load of data no thread writes during the kernel, at a wave-uniform address:
// a scalar load through the constant address space, ordered by the scalar
// memory counter rather than behind the wave's outstanding vector loads and
// stores.
template <typename T>
__device__ __forceinline__ T ld_uniform(const T* p) {
    return *(const __attribute__((address_space(4))) T*)p;
}

__device__ __forceinline__ int tid_local() {
    int t = threadIdx.x;
    asm volatile("" : "+v"(t));
    return t;
}

// ---------------------------------------------------------------------------
// Accesses to data that other workgroups of the same launch produce or consume
// (COH = true): device scope, so loads never hit a stale line of another XCD's
// L2 and stores are visible device-wide once they complete.  With COH = false
// they are ordinary accesses (data crosses kernel boundaries only).
// ---------------------------------------------------------------------------
template <bool COH>
__device__ __forceinline__ float ld_f32(const float* p) {
    if (COH) return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return *p;
}
template <bool COH>
__device__ __forceinline__ void st_f32(float* p, float v) {
    if (COH)
        __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else
        *p = v;
}
template <bool COH>
__device__ __forceinline__ void st_u16(uint16_t* p, uint16_t v) {
    if (COH)
        __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else
        *p = v;
}
// 16 bytes (16-byte aligned)
template <bool COH>
__device__ __forceinline__ u32x4 ld_16B(const void* p) {
    if (COH) {
        const unsigned long long* q = (const unsigned long long*)p;
        const unsigned long long a = __hip_atomic_load(q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const unsigned long long b = __hip_atomic_load(q + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return u32x4{(unsigned)a, (unsigned)(a >> 32), (unsigned)b, (unsigned)(b >> 32)};
    }
    return *(const u32x4*)p;
}

// ---------------------------------------------------------------------------
// Cross-lane reductions inside rows of 16 lanes by DPP moves (no LDS round
// trip).  Every lane of a group ends with the same value (IEEE addition is
// commutative).
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
// sum over aligned groups of L lanes (L = 1, 2, 4, 8 or 16)
template <int L>
__device__ __forceinline__ float group_sum(float v) {
    if (L >= 2) v += dpp_mov<0xB1>(v);      // quad_perm [1,0,3,2]
    if (L >= 4) v += dpp_mov<0x4E>(v);      // quad_perm [2,3,0,1]
    if (L >= 8) v += dpp_mov<0x141>(v);     // row_half_mirror
    if (L >= 16) v += dpp_mov<0x140>(v);    // row_mirror
    return v;
}
// ---------------------------------------------------------------------------
// 16-bit types.  bf16 is the type of the model's weights as given; the
// kernels compute with fp16 (11 significant bits against bf16's 8, the same
// two bytes): the packed weight copies, the activations that feed the GEMMs,
// the key/value caches and the attention products are fp16 with fp32
// accumulation.  A bf16 weight converts to fp16 exactly when its magnitude
// lies in [2^-17, 65504] (below, to the nearest fp16, off by < 2^-25).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }
// fp16 <-> fp32, round to nearest even
__device__ __forceinline__ float h2f(uint16_t b) { return (float)__builtin_bit_cast(_Float16, b); }
__device__ __forceinline__ uint16_t f2h(float f) { return __builtin_bit_cast(uint16_t, (_Float16)f); }
__device__ __forceinline__ uint32_t pack_h2(float a, float b) {
    return (uint32_t)f2h(a) | ((uint32_t)f2h(b) << 16);
}
constexpr float kF16Max = 65504.0f;

// ---------------------------------------------------------------------------
// Data-driven exchange inside the persistent pass.  Every activation buffer
// the pass exchanges between workgroups is filled with the sentinel pattern
// (all bits set) before the launch and written once during it; producers never
// store the sentinel (an all-ones NaN becomes the canonical quiet NaN), and
// consumers read with device-scope loads until no element is the sentinel.
// A read that does not see its data within the spin budget sets kErrPoll in
// the error word, and once that bit is set no read waits any more, so the
// launch always ends.
// ---------------------------------------------------------------------------
constexpr uint32_t kSentinel = 0xFFFFFFFFu;
constexpr int32_t kErrPoll = 8;
constexpr unsigned kPollSpin = 1u << 16;

__device__ __forceinline__ uint16_t h_value(float v) {
    const uint16_t b = f2h(v);
    return b == 0xFFFFu ? (uint16_t)0x7E00u : b;
}
__device__ __forceinline__ float f_value(float v) {
    return __float_as_uint(v) == kSentinel ? __uint_as_float(0x7FC00000u) : v;
}
// Some element of 16 bytes is the sentinel: the element-wise maximum over the
// four words (packed 16-bit maxima for fp16) reaches all ones exactly then.
// Consumers test every fragment of every poll round, so the test is a few
// instructions rather than one compare per element.
typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ bool sentinel16(const u32x4& u) {
    const u16x2 m = __builtin_elementwise_max(
        __builtin_elementwise_max(__builtin_bit_cast(u16x2, u[0]), __builtin_bit_cast(u16x2, u[1])),
        __builtin_elementwise_max(__builtin_bit_cast(u16x2, u[2]), __builtin_bit_cast(u16x2, u[3])));
    return __builtin_elementwise_max(m.x, m.y) == 0xFFFFu;
}
__device__ __forceinline__ bool sentinel32(const u32x4& u) {
    const uint32_t a = u[0] > u[1] ? u[0] : u[1], b = u[2] > u[3] ? u[2] : u[3];
    return (a > b ? a : b) == kSentinel;
}
// true once the launch gave up waiting (checked every 64 polls)
__device__ __forceinline__ bool poll_abort(unsigned n, int32_t* err) {
    if (n > kPollSpin) {
        atomicOr(err, kErrPoll);
        return true;
    }
    return (n & 63) == 63 && (__hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & kErrPoll);
}
// a device-scope fp32 value, once its producer has written it
__device__ __forceinline__ float poll_f32(const float* p, int32_t* err) {
    float v = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    for (unsigned n = 0; __float_as_uint(v) == kSentinel; ++n) {
        if (poll_abort(n, err)) break;
        __builtin_amdgcn_s_sleep(1);
        v = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    return v;
}
// 16 device-scope bytes (bf16 or fp32 elements), once no element is the sentinel
template <bool BF16>
__device__ __forceinline__ u32x4 poll_16B(const void* p, int32_t* err) {
    u32x4 u = ld_16B<true>(p);
    for (unsigned n = 0; BF16 ? sentinel16(u) : sentinel32(u); ++n) {
        if (poll_abort(n, err)) break;
        __builtin_amdgcn_s_sleep(1);
        u = ld_16B<true>(p);
    }
    return u;
}

// ---------------------------------------------------------------------------
// Row descriptor: one branch (or one prefill position) in a batched pass.
//   xrow   : row of the hidden-state array X this row reads and updates
//   slot   : branch slot owning the row's KV (its own position), or -1 for a
//            prefill position whose KV goes straight to the committed cache
//   seq    : sequence
//   pos    : position of the row's token
//   depth  : recurrent depth computed in this pass (core 1..R; the readout
//            depth for coda rows; 0 for prelude rows)
//   tdone  : positions < tdone are read from the sequence's committed cache
//   src    : X row a readout copy starts from (coda rows)
//   anc    : slots holding positions tdone .. pos-1 (the in-flight ancestors)
// ---------------------------------------------------------------------------
struct Row {
    int32_t xrow, slot, seq, pos, depth, tdone, src, pad;
    int32_t anc[kChainMax];
};

// ---------------------------------------------------------------------------
// Model / pool geometry (fixed for a handle)
// ---------------------------------------------------------------------------
struct Geo {
    int h, H, dh, F, V;
    int Lp, Lb, Lc;          // prelude / core / coda block counts
    int R;
    int T;                   // KV tables per position: Lp + R*Lb + R*Lc
    int max_ctx;
    int S;                   // branch slots
    int ssq_tiles;           // h / 16
    float eps;
    float attn_scale;        // 1/sqrt(dh)
};

enum Stack { STACK_PRE = 0, STACK_CORE = 1, STACK_CODA = 2 };

// KV table index of (stack, layer) at a row's depth
__device__ __host__ __forceinline__ int kv_table(const Geo& g, int stack, int layer, int depth) {
    if (stack == STACK_PRE) return layer;
    if (stack == STACK_CORE) return g.Lp + (depth - 1) * g.Lb + layer;
    return g.Lp + g.R * g.Lb + (depth - 1) * g.Lc + layer;
}
// committed cache, head-major: [seq][T][2][H][max_ctx][dh] (one head's keys or
// values of consecutive positions are contiguous); offset of (head, pos)
__device__ __host__ __forceinline__ size_t kvc_index(const Geo& g, int seq, int t, int kv, int head, int pos) {
    return (((((size_t)seq * g.T + t) * 2 + kv) * g.H + head) * (size_t)g.max_ctx + pos) * (size_t)g.dh;
}
// slot cache: [slot][T][2][h]
__device__ __host__ __forceinline__ size_t kvs_index(const Geo& g, int slot, int t, int kv) {
    return (((size_t)slot * g.T + t) * 2 + kv) * (size_t)g.h;
}

// sum of squares of 16 consecutive values, in index order: the partial that
// every writer of a pass row stores per 16-column tile (RMSNorm statistics)
__device__ __forceinline__ float ssq16(const float* v) {
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 16; ++j) s = fmaf(v[j], v[j], s);
    return s;
}

// Pass buffers, in row order of the pass's row list:
//   XB   [rows][h]         hidden state rounded to the weight dtype (GEMM A operand)
//   SSQR [rows][h/16]      sums of squares per 16-column tile of the fp32 state
struct PassBuf {
    void* XB;
    float* SSQR;
};

}  // namespace ls
