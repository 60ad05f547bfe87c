// Device-side attention pieces (one kChunk-position chunk of one (row, head) per
// wave, and the chunk-order combination), shared by the standalone attention
// kernel (ls_attn.hip) and the persistent pass kernel (ls_pass.hip).
#pragma once
#include "ls_attn.h"
#include "ls_gemm_dev.h"   // buffer resources

namespace ls {

template <typename WT>
struct KV;
template <>
struct KV<uint16_t> {
    static constexpr int E = 8;                   // fp16 elements per 16 bytes
    __device__ static void unpack(const u32x4& u, float* v) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            v[2 * e] = h2f((uint16_t)(u[e] & 0xFFFFu));
            v[2 * e + 1] = h2f((uint16_t)(u[e] >> 16));
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

// Softmax arithmetic works in base 2: scores are scaled by attn_scale * log2(e)
// and weights are exp2 of score differences (v_exp_f32), which equals the
// natural-base softmax; maxima and sums pass between partials in these units.
constexpr float kLog2e = 1.4426950408889634f;
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// fp16 pair dot product accumulated in fp32 (v_dot2_f32_f16): acc + a.lo*b.lo + a.hi*b.hi
__device__ __forceinline__ float dot2_f16(uint32_t a, uint32_t b, float acc) {
    return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, a), __builtin_bit_cast(f16x2, b), acc, false);
}

// Address of one head's keys (kv = 0) or values (kv = 1) at one position of a row.
template <typename WT>
__device__ __forceinline__ const WT* kv_row(const AttnParams& p, const Row& row, const int* anc, int t, int kv,
                                            int head, int pos) {
    if (row.slot < 0 || pos < row.tdone) return (const WT*)p.kvc + kvc_index(p.g, row.seq, t, kv, head, pos);
    const int s = pos < row.pos ? anc[pos - row.tdone] : row.slot;
    return (const WT*)p.kvs + kvs_index(p.g, s, t, kv) + head * p.g.dh;
}

// 16 bytes of keys (kv = 0) or values (kv = 1) of one position.  COH: the
// row's own position is written by another workgroup of the same launch, so it
// is read at device scope; every other position was written by earlier
// launches.
template <typename WT, bool COH>
__device__ __forceinline__ u32x4 kv_load(const AttnParams& p, const Row& row, const int* anc, int t, int kv, int head,
                                         int pos, int off) {
    const WT* a = kv_row<WT>(p, row, anc, t, kv, head, pos) + off;
    if (COH && pos == row.pos) return ld_16B<true>(a);
    return *(const u32x4*)a;
}

// sum / max over the lanes with the same index modulo L (L = 2 .. 32)
template <int L, bool MAX>
__device__ __forceinline__ float across_groups(float v) {
#pragma unroll
    for (int o = L; o < 64; o <<= 1) {
        float u;
        if (o == 2) u = dpp_mov<0x4E>(v);           // quad_perm [2,3,0,1]
        else if (o == 4) u = dpp_mov<0x124>(v);     // row_ror:4
        else if (o == 8) u = dpp_mov<0x128>(v);     // row_ror:8
        else u = __shfl_xor(v, o);
        v = MAX ? fmaxf(v, u) : v + u;
    }
    return v;
}

// value of lane `l` (wave-uniform index) as a scalar broadcast
__device__ __forceinline__ float lane_read(float v, int l) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}

// Lane geometry of a head slice: a position's DH values are LPP lanes x 16
// bytes (E elements each), so one load instruction covers PPI = 64/LPP whole
// positions and a chunk of kChunk positions takes NIT instructions for the keys and
// NIT for the values (few cache lines per instruction).
template <typename WT, int DH>
struct AttnGeo {
    static constexpr int E = KV<WT>::E;
    static constexpr int NK = DH / E;                  // 16-byte vectors per head slice
    static_assert(NK <= 16, "a head slice must fit 16 lanes");
    static constexpr int LPP = NK <= 2 ? 2 : NK <= 4 ? 4 : NK <= 8 ? 8 : 16;
    static constexpr int PPI = 64 / LPP, NIT = kChunk / PPI;
};

// Header fields of row m (its chain of ancestors stays in memory).
__device__ __forceinline__ Row row_head(const Row* rows, int m) {
    Row r;
    r.slot = rows[m].slot;
    r.seq = rows[m].seq;
    r.pos = rows[m].pos;
    r.depth = rows[m].depth;
    r.tdone = rows[m].tdone;
    return r;
}

// Keys and values of a chunk wholly below the sequence's committed length:
// 64 consecutive positions of one head, one contiguous block of keys and one
// of values (lanes past the head slice read zero).  Uniform arguments.
template <typename WT, int DH>
__device__ __forceinline__ void chunk_kv_committed(const AttnParams& p, int seq, int t, int head, int p0,
                                                   u32x4 (&kr)[AttnGeo<WT, DH>::NIT],
                                                   u32x4 (&vr)[AttnGeo<WT, DH>::NIT]) {
    using A = AttnGeo<WT, DH>;
    constexpr int E = A::E, NIT = A::NIT, PPI = A::PPI, LPP = A::LPP;
    const int lane = tid_local() & 63;
    const int d8 = lane % LPP, grp = lane / LPP;
    const bool dv = d8 < A::NK;
    const int off = d8 * E;
    constexpr int pstride = DH * (int)sizeof(WT);
    const __amdgpu_buffer_rsrc_t rk =
        buf_rsrc((const WT*)p.kvc + kvc_index(p.g, seq, t, 0, head, p0), (uint32_t)(kChunk * pstride));
    const __amdgpu_buffer_rsrc_t rv =
        buf_rsrc((const WT*)p.kvc + kvc_index(p.g, seq, t, 1, head, p0), (uint32_t)(kChunk * pstride));
    const int lofs = dv ? grp * pstride + off * (int)sizeof(WT) : kOutOfRange;
#pragma unroll
    for (int it = 0; it < NIT; ++it) kr[it] = buf_load16<0>(rk, lofs, it * PPI * pstride);
#pragma unroll
    for (int it = 0; it < NIT; ++it) vr[it] = buf_load16<0>(rv, lofs, it * PPI * pstride);
}

template <typename WT, int DH>
__device__ __forceinline__ void chunk_math(const AttnParams& p, const u32x4 (&qr)[KV<WT>::E / 4],
                                           const u32x4 (&kr)[AttnGeo<WT, DH>::NIT],
                                           const u32x4 (&vr)[AttnGeo<WT, DH>::NIT], int p0, int plast,
                                           float (&acc)[KV<WT>::E], float& mx_out, float& l_out);

// Partial of chunk c (positions kChunk*c .. kChunk*c + kChunk - 1, clipped to
// plast: the row's own position, or the one before it) of one (row, head) by
// the calling wave: the softmax-weighted value
// sum (dims d8*E .. d8*E+E-1, identical in every lane with the same d8), the
// chunk's score maximum and its weight sum.  A score reduces over the LPP
// lanes of its position; each lane then holds the weights of exactly the
// positions its value registers hold.  The query (row m) is requested before
// the keys and values.  COH (persistent pass): the query and the row's own
// keys / values are produced in the same launch and read until written.
template <typename WT, int DH, bool COH>
__device__ __forceinline__ void attn_chunk(const AttnParams& p, const Row& row_in, int m, const int* anc, int t,
                                           int head, int c, int plast, float (&acc)[KV<WT>::E], float& mx_out,
                                           float& l_out) {
    using A = AttnGeo<WT, DH>;
    constexpr int E = A::E, NIT = A::NIT, PPI = A::PPI, LPP = A::LPP;
    // every argument is the same in all lanes: keep it in scalar registers, so
    // the buffer resources below need no per-lane waterfall
    Row row;
    row.slot = __builtin_amdgcn_readfirstlane(row_in.slot);
    row.seq = __builtin_amdgcn_readfirstlane(row_in.seq);
    row.pos = __builtin_amdgcn_readfirstlane(row_in.pos);
    row.depth = __builtin_amdgcn_readfirstlane(row_in.depth);
    row.tdone = __builtin_amdgcn_readfirstlane(row_in.tdone);
    m = __builtin_amdgcn_readfirstlane(m);
    t = __builtin_amdgcn_readfirstlane(t);
    head = __builtin_amdgcn_readfirstlane(head);
    c = __builtin_amdgcn_readfirstlane(c);
    plast = __builtin_amdgcn_readfirstlane(plast);
    const int lane = tid_local() & 63;
    const int d8 = lane % LPP, grp = lane / LPP;
    const bool dv = d8 < A::NK;
    const int off = d8 * E;                            // within the head slice
    const int p0 = c * kChunk;
    // the query first: scores can start as soon as the first keys arrive
    // (loads complete in issue order)
    const float* qsrc = p.q + (size_t)m * p.g.h + head * DH + off;
    u32x4 qr[E / 4];
#pragma unroll
    for (int e = 0; e < E / 4; ++e) qr[e] = dv ? ld_16B<COH>(qsrc + 4 * e) : u32x4{0u, 0u, 0u, 0u};
    u32x4 kr[NIT], vr[NIT];
    if (p0 + kChunk <= row.tdone) {
        chunk_kv_committed<WT, DH>(p, row.seq, t, head, p0, kr, vr);
    } else {
#pragma unroll
        for (int it = 0; it < NIT; ++it) {
            const int ps = p0 + it * PPI + grp;
            kr[it] = (ps <= plast && dv) ? kv_load<WT, COH>(p, row, anc, t, 0, head, ps, off)
                                           : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int it = 0; it < NIT; ++it) {
            const int ps = p0 + it * PPI + grp;
            vr[it] = (ps <= plast && dv) ? kv_load<WT, COH>(p, row, anc, t, 1, head, ps, off)
                                           : u32x4{0u, 0u, 0u, 0u};
        }
        if (COH) {
            // the row's own keys / values come from this launch's QKV phase
#pragma unroll
            for (int it = 0; it < NIT; ++it) {
                const int ps = p0 + it * PPI + grp;
                if (ps != row.pos || !dv) continue;
                constexpr bool BF = sizeof(WT) == 2;
                if (BF ? sentinel16(kr[it]) : sentinel32(kr[it]))
                    kr[it] = poll_16B<BF>(kv_row<WT>(p, row, anc, t, 0, head, ps) + off, p.err);
                if (BF ? sentinel16(vr[it]) : sentinel32(vr[it]))
                    vr[it] = poll_16B<BF>(kv_row<WT>(p, row, anc, t, 1, head, ps) + off, p.err);
            }
        }
    }
#pragma unroll
    for (int e = 0; e < E / 4; ++e)
        if (COH && dv && sentinel32(qr[e])) qr[e] = poll_16B<false>(qsrc + 4 * e, p.err);
    chunk_math<WT, DH>(p, qr, kr, vr, p0, plast, acc, mx_out, l_out);
}

// The partial of one chunk from its query, keys and values in registers
// (lanes laid out as AttnGeo; positions past plast weigh nothing).
template <typename WT, int DH>
__device__ __forceinline__ void chunk_math(const AttnParams& p, const u32x4 (&qr)[KV<WT>::E / 4],
                                           const u32x4 (&kr)[AttnGeo<WT, DH>::NIT],
                                           const u32x4 (&vr)[AttnGeo<WT, DH>::NIT], int p0, int plast,
                                           float (&acc)[KV<WT>::E], float& mx_out, float& l_out) {
    using A = AttnGeo<WT, DH>;
    constexpr int E = A::E, NIT = A::NIT, PPI = A::PPI, LPP = A::LPP;
    const int lane = tid_local() & 63;
    const int grp = lane / LPP;
    float qf[E];
#pragma unroll
    for (int e = 0; e < E / 4; ++e)
#pragma unroll
        for (int j = 0; j < 4; ++j) qf[4 * e + j] = __uint_as_float(qr[e][j]);
    const float sl2 = p.g.attn_scale * kLog2e;
    float sc[NIT];
    float mx = -INFINITY;
    float l = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = 0.f;
    if constexpr (sizeof(WT) == 2) {
        // fp16 keys and values: the query is rounded to fp16 pairs once and
        // every product runs as an fp16 pair dot product (v_dot2) into fp32;
        // the weights of two positions (rounded to fp16) meet the values of
        // those positions, paired per dimension, the same way
        uint32_t qb[E / 2];
#pragma unroll
        for (int k = 0; k < E / 2; ++k) qb[k] = pack_h2(qf[2 * k], qf[2 * k + 1]);
#pragma unroll
        for (int it = 0; it < NIT; ++it) {
            float s = 0.f;
#pragma unroll
            for (int k = 0; k < E / 2; ++k) s = dot2_f16(qb[k], kr[it][k], s);
            s = group_sum<LPP>(s);
            sc[it] = (p0 + it * PPI + grp <= plast) ? s * sl2 : -INFINITY;
            mx = fmaxf(mx, sc[it]);
        }
        mx = across_groups<LPP, true>(mx);
#pragma unroll
        for (int it = 0; it < NIT; it += 2) {
            const float w0 = (p0 + it * PPI + grp <= plast) ? exp2_fast(sc[it] - mx) : 0.f;
            const float w1 = (p0 + (it + 1) * PPI + grp <= plast) ? exp2_fast(sc[it + 1] - mx) : 0.f;
            const uint32_t wp = pack_h2(w0, w1);
            l += h2f((uint16_t)(wp & 0xFFFFu));
            l += h2f((uint16_t)(wp >> 16));
#pragma unroll
            for (int k = 0; k < E / 2; ++k) {
                const uint32_t a = vr[it][k], b = vr[it + 1][k];
                acc[2 * k] = dot2_f16(wp, __builtin_amdgcn_perm(b, a, 0x05040100u), acc[2 * k]);
                acc[2 * k + 1] = dot2_f16(wp, __builtin_amdgcn_perm(b, a, 0x07060302u), acc[2 * k + 1]);
            }
        }
    } else {
#pragma unroll
        for (int it = 0; it < NIT; ++it) {
            float kf[E];
            KV<WT>::unpack(kr[it], kf);
            float s = 0.f;
#pragma unroll
            for (int e = 0; e < E; ++e) s = fmaf(qf[e], kf[e], s);
            s = group_sum<LPP>(s);
            sc[it] = (p0 + it * PPI + grp <= plast) ? s * sl2 : -INFINITY;
            mx = fmaxf(mx, sc[it]);
        }
        mx = across_groups<LPP, true>(mx);
#pragma unroll
        for (int it = 0; it < NIT; ++it) {
            const float w = (p0 + it * PPI + grp <= plast) ? exp2_fast(sc[it] - mx) : 0.f;
            l += w;
            float vf[E];
            KV<WT>::unpack(vr[it], vf);
#pragma unroll
            for (int e = 0; e < E; ++e) acc[e] = fmaf(w, vf[e], acc[e]);
        }
    }
    l = across_groups<LPP, false>(l);
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = across_groups<LPP, false>(acc[e]);
    mx_out = mx;
    l_out = l;
}

// Partial of the row's own position alone (a one-position chunk): maximum =
// its score, weight sum 1, weighted values = its values.  COH: the key, value
// and query come from this launch's QKV phase and are read until written.
template <typename WT, int DH, bool COH>
__device__ __forceinline__ void attn_own(const AttnParams& p, const Row& row_in, int m, const int* anc, int t,
                                         int head, float (&acc)[KV<WT>::E], float& mx_out, float& l_out) {
    using A = AttnGeo<WT, DH>;
    constexpr int E = A::E, LPP = A::LPP;
    constexpr bool BF = sizeof(WT) == 2;
    Row row;
    row.slot = __builtin_amdgcn_readfirstlane(row_in.slot);
    row.seq = __builtin_amdgcn_readfirstlane(row_in.seq);
    row.pos = __builtin_amdgcn_readfirstlane(row_in.pos);
    row.depth = __builtin_amdgcn_readfirstlane(row_in.depth);
    row.tdone = __builtin_amdgcn_readfirstlane(row_in.tdone);
    m = __builtin_amdgcn_readfirstlane(m);
    t = __builtin_amdgcn_readfirstlane(t);
    head = __builtin_amdgcn_readfirstlane(head);
    const int d8 = (tid_local() & 63) % LPP;
    const bool dv = d8 < A::NK;
    const int off = d8 * E;
    const float* qsrc = p.q + (size_t)m * p.g.h + head * DH + off;
    u32x4 qr[E / 4];
#pragma unroll
    for (int e = 0; e < E / 4; ++e) qr[e] = dv ? ld_16B<COH>(qsrc + 4 * e) : u32x4{0u, 0u, 0u, 0u};
    u32x4 kr = dv ? kv_load<WT, COH>(p, row, anc, t, 0, head, row.pos, off) : u32x4{0u, 0u, 0u, 0u};
    u32x4 vr = dv ? kv_load<WT, COH>(p, row, anc, t, 1, head, row.pos, off) : u32x4{0u, 0u, 0u, 0u};
    if (COH && dv) {
        if (BF ? sentinel16(kr) : sentinel32(kr)) kr = poll_16B<BF>(kv_row<WT>(p, row, anc, t, 0, head, row.pos) + off, p.err);
        if (BF ? sentinel16(vr) : sentinel32(vr)) vr = poll_16B<BF>(kv_row<WT>(p, row, anc, t, 1, head, row.pos) + off, p.err);
#pragma unroll
        for (int e = 0; e < E / 4; ++e)
            if (sentinel32(qr[e])) qr[e] = poll_16B<false>(qsrc + 4 * e, p.err);
    }
    float qf[E];
#pragma unroll
    for (int e = 0; e < E / 4; ++e)
#pragma unroll
        for (int j = 0; j < 4; ++j) qf[4 * e + j] = __uint_as_float(qr[e][j]);
    KV<WT>::unpack(vr, acc);
    float s = 0.f;
    if constexpr (sizeof(WT) == 2) {   // the same fp16 pair products as the chunks
#pragma unroll
        for (int k = 0; k < E / 2; ++k) s = dot2_f16(pack_h2(qf[2 * k], qf[2 * k + 1]), kr[k], s);
    } else {
        float kf[E];
        KV<WT>::unpack(kr, kf);
#pragma unroll
        for (int e = 0; e < E; ++e) s = fmaf(qf[e], kf[e], s);
    }
    mx_out = group_sum<LPP>(s) * (p.g.attn_scale * kLog2e);
    l_out = 1.f;
}

template <typename WT, int DH, bool COH>
__device__ __forceinline__ void attn_combine_lds(const AttnParams& p, int m, int head, int n, const float* smem);

// One (row m, head) item by the whole workgroup: its waves take the chunks of
// the positions before the row's own, then the own position as one more
// partial (so a row at position 512 fills 8 waves with 8 full chunks); the
// partials are combined in LDS in chunk order.  COH: inside the persistent
// pass (device-scope query, own key / value and output).
// LDS: [chunks + 1][DH + 2] partials.
template <typename WT, int DH, bool COH>
__device__ __forceinline__ void attn_item(const AttnParams& p, int m, int head, float* smem) {
    using A = AttnGeo<WT, DH>;
    constexpr int E = A::E;
    const Row row = row_head(p.rows, m);
    const int* anc = p.rows[m].anc;
    const int tid = tid_local(), wave = tid >> 6, lane = tid & 63, W = blockDim.x >> 6;
    const int np = (row.pos + kChunk - 1) / kChunk, n = np + 1;
    const int t = kv_table(p.g, p.stack, p.layer, row.depth);
    const int d8 = lane % A::LPP, grp = lane / A::LPP;
    for (int c = wave; c < n; c += W) {
        float acc[E], mx, l;
        if (c < np)
            attn_chunk<WT, DH, COH>(p, row, m, anc, t, head, c, row.pos - 1, acc, mx, l);
        else
            attn_own<WT, DH, COH>(p, row, m, anc, t, head, acc, mx, l);
        float* dst = smem + c * (DH + 2);
        if (grp == 0 && d8 < A::NK) {
#pragma unroll
            for (int e = 0; e < E; ++e) dst[d8 * E + e] = acc[e];
        }
        if (lane == 0) {
            dst[DH] = mx;
            dst[DH + 1] = l;
        }
    }
    __syncthreads();
    attn_combine_lds<WT, DH, COH>(p, m, head, n, smem);
    __syncthreads();
}

// The output of (row m, head) from its n partials in LDS ([n][DH + 2]): every
// output dimension derives the chunk weights exp2(max_c - max) itself and
// sums its chunk values and the weight sums with them in chunk order
// (partials in groups of CB: every LDS read of a group is issued before any
// is used; partials past n read partial 0 and weigh nothing).
template <typename WT, int DH, bool COH>
__device__ __forceinline__ void attn_combine_lds(const AttnParams& p, int m, int head, int n, const float* smem) {
    const int tid = tid_local();
    constexpr int CB = 8;
    for (int d = tid; d < DH; d += blockDim.x) {
        float mx = -INFINITY;
        for (int c0 = 0; c0 < n; c0 += CB) {
            float v[CB];
#pragma unroll
            for (int i = 0; i < CB; ++i) v[i] = smem[(c0 + i < n ? c0 + i : 0) * (DH + 2) + DH];
#pragma unroll
            for (int i = 0; i < CB; ++i) mx = fmaxf(mx, v[i]);
        }
        float l = 0.f, o = 0.f;
        for (int c0 = 0; c0 < n; c0 += CB) {
            float vm[CB], vl[CB], vo[CB];
#pragma unroll
            for (int i = 0; i < CB; ++i) {
                const float* b = smem + (c0 + i < n ? c0 + i : 0) * (DH + 2);
                vm[i] = b[DH];
                vl[i] = b[DH + 1];
                vo[i] = b[d];
            }
#pragma unroll
            for (int i = 0; i < CB; ++i) {
                if (c0 + i >= n) break;
                const float w = exp2_fast(vm[i] - mx);
                l = fmaf(vl[i], w, l);
                o = fmaf(vo[i], w, o);
            }
        }
        const float r = o / l;
        const size_t idx = (size_t)m * p.g.h + head * DH + d;
        if (sizeof(WT) == 2)
            st_u16<COH>((uint16_t*)p.out + idx, COH ? h_value(r) : f2h(r));
        else
            st_f32<COH>((float*)p.out + idx, COH ? f_value(r) : r);
    }
}

// One part of a (row m, head) item of the persistent pass whose row has more
// partials n than the workgroup has waves: part `part` of `parts` computes
// partials part * W .. part * W + W - 1 (one per wave), stores them at device
// scope in gpart[(m * H + head) * (chunks_cap + 1) + c][DH + 2] and counts the
// part on cnt[m * H + head] (zero at launch, so layer l's parts complete it at
// (l + 1) * parts); the workgroup that completes it loads all n partials into
// LDS and combines them with attn_combine_lds, the arithmetic of attn_item, so
// a row's output does not depend on how its item was split.
template <typename WT, int DH>
__device__ __forceinline__ void attn_item_part(const AttnParams& p, int m, int head, int part, int parts, float* gpart,
                                               unsigned* cnt, float* smem) {
    using A = AttnGeo<WT, DH>;
    constexpr int E = A::E;
    const Row row = row_head(p.rows, m);
    const int* anc = p.rows[m].anc;
    const int tid = tid_local(), wave = tid >> 6, lane = tid & 63, W = blockDim.x >> 6;
    const int np = (row.pos + kChunk - 1) / kChunk, n = np + 1;
    const int t = kv_table(p.g, p.stack, p.layer, row.depth);
    const int d8 = lane % A::LPP, grp = lane / A::LPP;
    float* base = gpart + (size_t)(m * p.g.H + head) * (p.chunks_cap + 1) * (DH + 2);
    const int c = part * W + wave;
    if (c < n) {
        float acc[E], mx, l;
        if (c < np)
            attn_chunk<WT, DH, true>(p, row, m, anc, t, head, c, row.pos - 1, acc, mx, l);
        else
            attn_own<WT, DH, true>(p, row, m, anc, t, head, acc, mx, l);
        float* dst = base + (size_t)c * (DH + 2);
        if (grp == 0 && d8 < A::NK) {
#pragma unroll
            for (int e = 0; e < E; ++e) st_f32<true>(dst + d8 * E + e, acc[e]);
        }
        if (lane == 0) {
            st_f32<true>(dst + DH, mx);
            st_f32<true>(dst + DH + 1, l);
        }
    }
    __builtin_amdgcn_s_waitcnt(0);                      // this wave's partial is visible device-wide
    __syncthreads();
    // the flag word sits past the n partials (the region holds chunks_cap + 1 of DH + 3 words)
    int* flag = (int*)(smem + (size_t)(p.chunks_cap + 1) * (DH + 2));
    if (tid == 0) {
        const unsigned old =
            __hip_atomic_fetch_add(cnt + m * p.g.H + head, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        *flag = old + 1 == (unsigned)((p.layer + 1) * parts);
    }
    __syncthreads();
    const bool lastp = *flag != 0;
    __syncthreads();
    if (!lastp) return;
    for (int i = tid; i < n * (DH + 2); i += blockDim.x) smem[i] = ld_f32<true>(base + i);
    __syncthreads();
    attn_combine_lds<WT, DH, true>(p, m, head, n, smem);
    __syncthreads();
}

// Attention phase of the persistent pass: tasks (row, head, chunk) in row
// order, task k on wave (k / G) % W of workgroup slot k % G, so the key/value
// stream spreads over every CU.  Each wave stores its chunk partial (device
// scope) in part[(m*H + head)*chunks_cap + c][DH+2] and counts it on
// cnt[m*H + head]; the wave that completes a (row, head) -- the count reaching
// (layer + 1) * chunks, the counters being zero at launch -- combines the
// partials in chunk order (the arithmetic of attn_combine, with every partial
// loaded up front) and writes the output row slice.  At most 128 chunks.
template <typename WT, int DH>
__device__ __forceinline__ void attn_tasks(const AttnParams& p, int M, int slot, int G, float* part, unsigned* cnt) {
    using A = AttnGeo<WT, DH>;
    constexpr int E = A::E, DPL = (DH + 63) / 64, CB = 16;
    const int tid = tid_local(), wave = tid >> 6, lane = tid & 63, W = blockDim.x >> 6;
    const int H = p.g.H, cap = p.chunks_cap;
    // per-row task counts and their inclusive prefix (one row per lane)
    const int nl = lane < M ? p.rows[lane].pos / kChunk + 1 : 0;
    int pre = nl * H;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int v = __shfl_up(pre, o);
        if (lane >= o) pre += v;
    }
    const int total = __shfl(pre, 63);
    const int d8 = lane % A::LPP, grp = lane / A::LPP;
    for (int k = slot + G * wave; k < total; k += G * W) {
        // row of task k: the number of rows whose prefix is <= k
        const int m = __popcll(__ballot(lane < M && pre <= k));
        const int before = m ? __shfl(pre, m - 1) : 0;
        const int n = __shfl(nl, m);
        const int r = k - before, head = r / n, c = r - head * n;
        const Row row = row_head(p.rows, m);
        const int t = kv_table(p.g, p.stack, p.layer, row.depth);
        float acc[E], mx, l;
        attn_chunk<WT, DH, true>(p, row, m, p.rows[m].anc, t, head, c, row.pos, acc, mx, l);
        float* base = part + (size_t)(m * H + head) * cap * (DH + 2);
        float* dst = base + (size_t)c * (DH + 2);
        if (grp == 0 && d8 < A::NK) {
#pragma unroll
            for (int e = 0; e < E; ++e) st_f32<true>(dst + d8 * E + e, acc[e]);
        }
        if (lane == 0) {
            st_f32<true>(dst + DH, mx);
            st_f32<true>(dst + DH + 1, l);
        }
        __builtin_amdgcn_s_waitcnt(0);                  // the partial is visible device-wide
        unsigned old = 0;
        if (lane == 0)
            old = __hip_atomic_fetch_add(cnt + m * H + head, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        old = __shfl(old, 0);
        if (old + 1 != (unsigned)((p.layer + 1) * n)) continue;
        // ---- last partial of (m, head): combine in chunk order ------------------
        // chunk statistics: chunk c in lane c % 64, register c / 64
        const float* st0 = base + (size_t)lane * (DH + 2) + DH;
        const float* st1 = st0 + (size_t)64 * (DH + 2);
        const float mc0 = lane < n ? ld_f32<true>(st0) : -INFINITY;
        const float lc0 = lane < n ? ld_f32<true>(st0 + 1) : 0.f;
        const float mc1 = lane + 64 < n ? ld_f32<true>(st1) : -INFINITY;
        const float lc1 = lane + 64 < n ? ld_f32<true>(st1 + 1) : 0.f;
        // every o partial of the first CB chunks is requested before any is used;
        // chunks past n contribute exact zeros (weight 0, value 0)
        float v[CB][DPL];
#pragma unroll
        for (int i = 0; i < CB; ++i)
#pragma unroll
            for (int j = 0; j < DPL; ++j) {
                const int d = lane + 64 * j;
                v[i][j] = (i < n && d < DH) ? ld_f32<true>(base + (size_t)i * (DH + 2) + d) : 0.f;
            }
        float gmx = fmaxf(mc0, mc1);
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) gmx = fmaxf(gmx, __shfl_xor(gmx, o));
        const float wc0 = lane < n ? exp2_fast(mc0 - gmx) : 0.f;
        const float wc1 = lane + 64 < n ? exp2_fast(mc1 - gmx) : 0.f;
        float lsum = 0.f, o[DPL];
#pragma unroll
        for (int j = 0; j < DPL; ++j) o[j] = 0.f;
        for (int c0 = 0; c0 < n; c0 += CB) {
            if (c0) {   // partials past the first CB chunks
#pragma unroll
                for (int i = 0; i < CB; ++i)
#pragma unroll
                    for (int j = 0; j < DPL; ++j) {
                        const int d = lane + 64 * j;
                        v[i][j] = (c0 + i < n && d < DH) ? ld_f32<true>(base + (size_t)(c0 + i) * (DH + 2) + d) : 0.f;
                    }
            }
#pragma unroll
            for (int i = 0; i < CB; ++i) {
                const int c = c0 + i;                   // wave-uniform: lane reads, no LDS
                const float w = c < n ? lane_read(c < 64 ? wc0 : wc1, c & 63) : 0.f;
                const float lcc = c < n ? lane_read(c < 64 ? lc0 : lc1, c & 63) : 0.f;
                lsum += lcc * w;
#pragma unroll
                for (int j = 0; j < DPL; ++j) o[j] += v[i][j] * w;
            }
        }
#pragma unroll
        for (int j = 0; j < DPL; ++j) {
            const int d = lane + 64 * j;
            if (d >= DH) break;
            const float rr = o[j] / lsum;
            const size_t idx = (size_t)m * p.g.h + head * DH + d;
            if (sizeof(WT) == 2)
                st_u16<true>((uint16_t*)p.out + idx, h_value(rr));
            else
                st_f32<true>((float*)p.out + idx, f_value(rr));
        }
    }
}

}  // namespace ls
