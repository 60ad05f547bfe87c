// Decode attention over per-depth KV caches.
//
// Computation at recurrent depth r needs the keys/values of the same depth
// (implementation details, KV cache management): a row at depth r and block
// layer l attends over positions 0..pos with the (r, l) cache.  Positions below
// the sequence's committed length come from the committed cache; positions of
// the row's in-flight ancestors come from their branch slots (a child reuses
// its parent's prefix instead of copying it); the row's own position comes from
// its own slot, written by the QKV epilogue of the same layer.
//
// One workgroup per (head, row).  Its wavefronts take 64-position chunks of
// *logical* position; inside a chunk each lane owns one key position (its dot
// product with the query needs no cross-lane reduction), every key load of the
// chunk is issued before any is used, then every value load.  Chunk partials
// (o, max, sum) stay in LDS and are combined in chunk order, so a row's result
// depends only on the values it reads, never on where they are stored or how
// many rows run: vanilla decoding and LoopSpec get bit-identical outputs.
#include "ls_attn.h"

namespace ls {

template <typename WT>
struct KV;
template <>
struct KV<uint16_t> {
    static constexpr int E = 8;                   // elements per 16 bytes
    __device__ static void unpack(const u32x4& u, float* v) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            v[2 * e] = __uint_as_float(u[e] << 16);
            v[2 * e + 1] = __uint_as_float(u[e] & 0xFFFF0000u);
        }
    }
};
template <>
struct KV<float> {
    static constexpr int E = 4;
    __device__ static void unpack(const u32x4& u, float* v) {
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = __uint_as_float(u[e]);
    }
};

// Address of the keys (kv = 0) or values (kv = 1) of one position of a row.
template <typename WT>
__device__ __forceinline__ const WT* kv_row(const AttnParams& p, const Row& row, const int* anc, int t, int kv,
                                            int pos) {
    if (row.slot < 0 || pos < row.tdone) return (const WT*)p.kvc + kvc_index(p.g, row.seq, t, kv, pos);
    const int s = pos < row.pos ? anc[pos - row.tdone] : row.slot;
    return (const WT*)p.kvs + kvs_index(p.g, s, t, kv);
}

// DH: head dim.  Keys: lane = position, DH/E 16-byte loads.  Values: LPP lanes
// per position, E dims each, 64/LPP positions per load instruction.
template <typename WT, int DH>
__global__ void __launch_bounds__(512) k_attn(AttnParams p) {
    constexpr int E = KV<WT>::E;
    constexpr int NK = DH / E;                         // key loads per lane
    constexpr int LPP = NK <= 2 ? 2 : NK <= 4 ? 4 : NK <= 8 ? 8 : 16;
    constexpr int PPI = 64 / LPP, NIT = kChunk / PPI;
    extern __shared__ float smem[];
    const int m = blockIdx.y;
    if (m >= *p.nrows) return;
    Row row;                                           // header fields only; the chain goes to LDS
    row.slot = p.rows[m].slot;
    row.seq = p.rows[m].seq;
    row.pos = p.rows[m].pos;
    row.depth = p.rows[m].depth;
    row.tdone = p.rows[m].tdone;
    const int head = blockIdx.x;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, W = blockDim.x >> 6;
    float* qs = smem;                                  // [DH]
    int* anc = (int*)(smem + DH);                      // [kChainMax]
    float* wts = smem + DH + kChainMax;                // [W][64] softmax weights
    float* part = wts + W * 64;                        // [chunks][DH + 2]
    for (int d = threadIdx.x; d < DH; d += blockDim.x) qs[d] = p.q[(size_t)m * p.g.h + head * DH + d];
    for (int i = threadIdx.x; i < kChainMax; i += blockDim.x) anc[i] = p.rows[m].anc[i];
    __syncthreads();
    const int n = row.pos / kChunk + 1;
    const int t = kv_table(p.g, p.stack, p.layer, row.depth);
    const int hoff = head * DH;
    const int d8 = lane % LPP, grp = lane / LPP;
    const bool dv = d8 < NK;
    for (int c = wave; c < n; c += W) {
        const int p0 = c * kChunk;
        // ---- scores: lane owns position p0 + lane ---------------------------
        const int kp = p0 + lane;
        const bool kval = kp <= row.pos;
        u32x4 kr[NK];
        {
            const WT* k = kval ? kv_row<WT>(p, row, anc, t, 0, kp) + hoff : nullptr;
#pragma unroll
            for (int i = 0; i < NK; ++i) kr[i] = kval ? *(const u32x4*)(k + i * E) : u32x4{0u, 0u, 0u, 0u};
        }
        // ---- values: issued before the scores are used ------------------------
        u32x4 vr[NIT];
#pragma unroll
        for (int it = 0; it < NIT; ++it) {
            const int vp = p0 + it * PPI + grp;
            vr[it] = (vp <= row.pos && dv) ? *(const u32x4*)(kv_row<WT>(p, row, anc, t, 1, vp) + hoff + d8 * E)
                                           : u32x4{0u, 0u, 0u, 0u};
        }
        float s = 0.f;
#pragma unroll
        for (int i = 0; i < NK; ++i) {
            float kf[E];
            KV<WT>::unpack(kr[i], kf);
#pragma unroll
            for (int e = 0; e < E; ++e) s = fmaf(qs[i * E + e], kf[e], s);
        }
        s = kval ? s * p.g.attn_scale : -INFINITY;
        float mx = s;
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
        const float w = kval ? expf(s - mx) : 0.f;
        float l = w;
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) l += __shfl_xor(l, o);
        wts[wave * 64 + lane] = w;
        __builtin_amdgcn_s_waitcnt(0xc07f);            // lgkmcnt(0): the weights are in LDS
        __builtin_amdgcn_wave_barrier();
        float acc[E];
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = 0.f;
#pragma unroll
        for (int it = 0; it < NIT; ++it) {
            const float wp = wts[wave * 64 + it * PPI + grp];
            float vf[E];
            KV<WT>::unpack(vr[it], vf);
#pragma unroll
            for (int e = 0; e < E; ++e) acc[e] = fmaf(wp, vf[e], acc[e]);
        }
#pragma unroll
        for (int o = LPP; o < 64; o <<= 1)
#pragma unroll
            for (int e = 0; e < E; ++e) acc[e] += __shfl_xor(acc[e], o);
        float* dst = part + c * (DH + 2);
        if (grp == 0 && dv) {
#pragma unroll
            for (int e = 0; e < E; ++e) dst[d8 * E + e] = acc[e];
        }
        if (lane == 0) {
            dst[DH] = mx;
            dst[DH + 1] = l;
        }
    }
    __syncthreads();
    for (int d = threadIdx.x; d < DH; d += blockDim.x) {
        float mx = -INFINITY;
        for (int c = 0; c < n; ++c) mx = fmaxf(mx, part[c * (DH + 2) + DH]);
        float l = 0.f, o = 0.f;
        for (int c = 0; c < n; ++c) {
            const float* b = part + c * (DH + 2);
            const float w = expf(b[DH] - mx);
            l += b[DH + 1] * w;
            o += b[d] * w;
        }
        const float r = o / l;
        const size_t idx = (size_t)m * p.g.h + hoff + d;
        if (sizeof(WT) == 2)
            ((uint16_t*)p.out)[idx] = f2bf(r);
        else
            ((float*)p.out)[idx] = r;
    }
}

int attention_waves(int chunks_cap) { return chunks_cap < 8 ? chunks_cap : 8; }

size_t attention_lds_bytes(int chunks_cap, int dh, int waves) {
    return ((size_t)dh + kChainMax + waves * 64 + (size_t)chunks_cap * (dh + 2)) * 4;
}

template <typename WT, int DH>
static void launch_dh(const AttnParams& p, int m_cap, hipStream_t st) {
    const int w = attention_waves(p.chunks_cap);
    hipLaunchKernelGGL((k_attn<WT, DH>), dim3(p.g.H, m_cap), dim3(64 * w), attention_lds_bytes(p.chunks_cap, DH, w),
                       st, p);
}

template <typename WT>
static hipError_t launch_t(const AttnParams& p, int m_cap, hipStream_t st) {
    switch (p.g.dh) {
        case 16: launch_dh<WT, 16>(p, m_cap, st); break;
        case 32: launch_dh<WT, 32>(p, m_cap, st); break;
        case 64: launch_dh<WT, 64>(p, m_cap, st); break;
        case 96: launch_dh<WT, 96>(p, m_cap, st); break;
        case 128: launch_dh<WT, 128>(p, m_cap, st); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <typename WT>
static hipError_t allow(int bytes) {
    const void* f[] = {(const void*)k_attn<WT, 16>, (const void*)k_attn<WT, 32>, (const void*)k_attn<WT, 64>,
                       (const void*)k_attn<WT, 96>, (const void*)k_attn<WT, 128>};
    for (const void* x : f) {
        hipError_t e = hipFuncSetAttribute(x, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t attention_prepare(int lds_bytes) {
    hipError_t e = allow<uint16_t>(lds_bytes);
    return e != hipSuccess ? e : allow<float>(lds_bytes);
}

hipError_t launch_attention(const AttnParams& p, bool bf16, int m_cap, hipStream_t st) {
    return bf16 ? launch_t<uint16_t>(p, m_cap, st) : launch_t<float>(p, m_cap, st);
}

}  // namespace ls
