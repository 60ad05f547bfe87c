// Device-side definitions shared by the LoopSpec gfx950 kernels and the host
// runtime that launches them.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ls {

// ---------------------------------------------------------------------------
// small vector types
// ---------------------------------------------------------------------------
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;

constexpr int kTile = 16;            // output features per MFMA tile (and per sum-of-squares partial)
constexpr int kMaxRows = 64;         // rows (branches) one batched pass handles
constexpr int kChunk = 64;           // attention positions per split-softmax chunk
constexpr int kChainMax = 24;        // in-flight ancestors a row can have (positions tdone .. pos-1)

// ---------------------------------------------------------------------------
// bf16 <-> fp32 (round to nearest even)
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }
__device__ __forceinline__ uint16_t f2bf(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}
__device__ __forceinline__ uint32_t pack_bf2(float a, float b) {
    return (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
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
// committed cache: [seq][T][2][max_ctx][h]
__device__ __host__ __forceinline__ size_t kvc_index(const Geo& g, int seq, int t, int kv, int pos) {
    return ((((size_t)seq * g.T + t) * 2 + kv) * (size_t)g.max_ctx + pos) * (size_t)g.h;
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
