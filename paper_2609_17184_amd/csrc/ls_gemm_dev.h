// Device-side pieces of the weight-streaming skinny GEMM, shared by the
// standalone GEMM kernels (ls_gemm.hip) and the persistent pass kernel
// (ls_pass.hip).  See ls_gemm.hip for the design.
#pragma once
#include "ls_gemm.h"

namespace ls {

template <typename WT>
struct WTraits;
template <>
struct WTraits<uint16_t> {
    static constexpr int KSTEP = 32;   // k values per 16-byte lane load
    static constexpr int VEC = 8;      // elements per 16 bytes
};
template <>
struct WTraits<float> {
    static constexpr int KSTEP = 16;
    static constexpr int VEC = 4;
};

// Row of the weight matrix feeding column j of a tile, and the matrix.
template <int EPI>
__device__ __forceinline__ int tile_row(const Geo& g, int tile, int j, int* mat) {
    if (EPI == EPI_QKV) {
        const int tph = g.h / kTile;                // tiles per matrix
        const int m = tile / tph, lt = tile - m * tph;
        const int tpd = g.dh / kTile;               // tiles per head
        const int head = lt / tpd, sub = lt - head * tpd;
        // columns j and j+8 hold a RoPE pair (i, i + dh/2)
        const int c = j < 8 ? sub * 8 + j : g.dh / 2 + sub * 8 + (j - 8);
        *mat = m;
        return head * g.dh + c;
    }
    *mat = 0;
    return tile * kTile + j;
}

template <typename WT, int NMAT>
__device__ __forceinline__ void mfma_step(const u32x4& a, const u32x4 (&b)[NMAT], f32x4 (&acc)[NMAT]) {
    if (sizeof(WT) == 2) {
        const f16x8 av = __builtin_bit_cast(f16x8, a);
#pragma unroll
        for (int q = 0; q < NMAT; ++q)
            acc[q] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, __builtin_bit_cast(f16x8, b[q]), acc[q], 0, 0, 0);
    } else {
        const f32x4 av = __builtin_bit_cast(f32x4, a);
#pragma unroll
        for (int q = 0; q < NMAT; ++q) {
            const f32x4 bb = __builtin_bit_cast(f32x4, b[q]);
#pragma unroll
            for (int e = 0; e < 4; ++e)
                acc[q] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[e], bb[e], acc[q], 0, 0, 0);
        }
    }
}

// Geometry of the calling wavefront inside work item `item` (a group of
// `tpw` tiles; one wave per (tile, k-slice)).  With k split over kg
// workgroups per tile, workgroup `kgi` of the tile holds the global slices
// kgi * ks .. kgi * ks + ks - 1 of the tile's ks * kg.
struct WaveGeo {
    int lane, wave, tl, ksl, tile, j, grp, nsteps, s0, nst;
    bool tile_ok;
};

__host__ __device__ __forceinline__ int gemm_kg(const GemmParams& p) { return p.kg > 1 ? p.kg : 1; }

template <typename WT, bool CONTIG>
__device__ __forceinline__ WaveGeo wave_geo(const GemmParams& p, int item, int kgi = 0) {
    WaveGeo w;
    const int tid = tid_local();
    w.lane = tid & 63;
    w.wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: scalar geometry
    w.tl = w.wave / p.ks;
    w.ksl = w.wave - w.tl * p.ks;
    w.tile = item * p.tpw + w.tl;
    w.tile_ok = w.tl < p.tpw && w.tile < p.tiles;
    w.j = w.lane & 15;
    w.grp = w.lane >> 4;
    w.nsteps = p.K / WTraits<WT>::KSTEP;
    if (CONTIG) {   // a contiguous block of steps per wave
        const unsigned KS = (unsigned)(p.ks * gemm_kg(p)), gs = (unsigned)(kgi * p.ks + w.ksl);
        w.s0 = (int)((unsigned)w.nsteps * gs / KS);
        w.nst = (int)((unsigned)w.nsteps * (gs + 1) / KS) - w.s0;
    } else {        // every ks-th step (all waves share staged activation chunks)
        w.s0 = 0;
        w.nst = w.ksl < w.nsteps ? (w.nsteps - w.ksl + p.ks - 1) / p.ks : 0;
    }
    return w;
}

// This wave's packed weight blocks: the tile's first block plus the lane offset.
template <typename WT, int NMAT>
__device__ __forceinline__ const WT* packed_tile(const GemmParams& p, const WaveGeo& w) {
    constexpr int VEC = WTraits<WT>::VEC;
    return (const WT*)p.Wp + (size_t)(w.tile_ok ? w.tile : 0) * w.nsteps * NMAT * 64 * VEC + w.lane * VEC;
}

// Buffer resource over [p, p + bytes): loads at offsets >= bytes return zero.
constexpr int kOutOfRange = (int)0x80000000u;   // a lane offset beyond every resource
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
// 16-byte buffer load; AUX 2 marks it nontemporal (streamed once), AUX 16
// gives it device scope (coherent with other workgroups' device-scope stores).
template <int AUX>
__device__ __forceinline__ u32x4 buf_load16(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, AUX));
}

// Weight registers of the direct path: every load of a wave in flight at once.
template <typename WT, int NMAT, int MAXS_>
struct BRegs {
    static constexpr int MAXS = MAXS_;
    u32x4 b[MAXS][NMAT];
};

// Issue the weight loads of the calling wave for `item` (direct path: the
// wave's steps must fit MAXS, which the launch configuration guarantees).
// The wave's blocks are contiguous (1 KB per step and matrix), so one scalar
// base plus constant offsets address them all.  Every register is loaded
// unconditionally: steps past the wave's share, waves without a tile and
// `live == false` read beyond the buffer range and get zeros, so no register
// keeps a value from an earlier phase and the MFMAs need no guards.
template <typename WT, int NMAT, int MAXS>
__device__ __forceinline__ void gemm_load_b(const GemmParams& p, int item, BRegs<WT, NMAT, MAXS>& R,
                                            bool live = true, int kgi = 0) {
    const WaveGeo w = wave_geo<WT, true>(p, item, kgi);
    const bool ok = live && w.tile_ok;
    const char* base = (const char*)p.Wp + (ok ? ((size_t)w.tile * w.nsteps + w.s0) * NMAT * 1024 : 0);
    const __amdgpu_buffer_rsrc_t rs = buf_rsrc(base, ok ? (uint32_t)w.nst * NMAT * 1024 : 0u);
    const int voff = w.lane * 16;
#pragma unroll
    for (int i = 0; i < MAXS; ++i) {
        const int vo = i < w.nst ? voff : kOutOfRange;
#pragma unroll
        for (int q = 0; q < NMAT; ++q) R.b[i][q] = buf_load16<2>(rs, vo, (i * NMAT + q) * 1024);
    }
}

// LDS staging of a wave's first kPfFrags weight fragments (1 KB each, in
// gemm_load_b's (step, matrix) order) for the work item of a later phase:
// direct-to-LDS buffer loads (each lane's 16 bytes land at lane * 16 of the
// fragment), issued while the workgroup still works on an earlier phase so the
// stream starts before the registers are free.  Steps past the wave's share
// land as zeros.  Loads complete in issue order, so once the wave has waited
// for any load issued after these, the staged fragments are in LDS.
constexpr int kPfFrags = 16;
template <typename WT, int NMAT, int MAXS>
__device__ __forceinline__ void gemm_stage_b(const GemmParams& p, int item, char* lds_wave) {
    const WaveGeo w = wave_geo<WT, true>(p, item);
    const bool ok = w.tile_ok;
    const char* base = (const char*)p.Wp + (ok ? ((size_t)w.tile * w.nsteps + w.s0) * NMAT * 1024 : 0);
    const __amdgpu_buffer_rsrc_t rs = buf_rsrc(base, ok ? (uint32_t)w.nst * NMAT * 1024 : 0u);
    const int voff = w.lane * 16;
#pragma unroll
    for (int j = 0; j < kPfFrags && j < MAXS * NMAT; ++j) {
        const int i = j / NMAT;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)(lds_wave + j * 1024),
                                                 16, i < w.nst ? voff : kOutOfRange, j * 1024, 0, 2);
    }
}

// gemm_load_b for an item whose first kPfFrags fragments gemm_stage_b staged
// in LDS: those come from LDS, the rest from memory.
template <typename WT, int NMAT, int MAXS>
__device__ __forceinline__ void gemm_load_b_staged(const GemmParams& p, int item, BRegs<WT, NMAT, MAXS>& R,
                                                   const char* lds_wave) {
    const WaveGeo w = wave_geo<WT, true>(p, item);
    const bool ok = w.tile_ok;
    const char* base = (const char*)p.Wp + (ok ? ((size_t)w.tile * w.nsteps + w.s0) * NMAT * 1024 : 0);
    const __amdgpu_buffer_rsrc_t rs = buf_rsrc(base, ok ? (uint32_t)w.nst * NMAT * 1024 : 0u);
    const int voff = w.lane * 16;
#pragma unroll
    for (int i = 0; i < MAXS; ++i) {
        const int vo = i < w.nst ? voff : kOutOfRange;
#pragma unroll
        for (int q = 0; q < NMAT; ++q) {
            const int j = i * NMAT + q;
            if (j < kPfFrags)
                R.b[i][q] = *(const __attribute__((address_space(3))) u32x4*)(lds_wave + j * 1024 + voff);
            else
                R.b[i][q] = buf_load16<2>(rs, vo, j * 1024);
        }
    }
}

// 1/rms of the rows (RMSNorm), cross-wave reduction of the accumulators in
// k-slice order, and the epilogue of the kind.  `ssv` holds the first
// NSS partials of row `wave` (loaded early by the caller).  When has_pre, the
// caller also loaded this thread's first-iteration operand early: RESID
// pre.x = residual value, QKV pre = (cos, sin) of its RoPE pair.  COH: activations
// are exchanged with other workgroups of the same launch (device-scope
// accesses).
//
// Split k (kg > 1, direct path, one tile per workgroup): the workgroup sums
// its slices in slice order and stores that partial (device scope); the last
// of the tile's kg workgroups to count itself on cnt[tile] (which it resets
// to zero for the next launch) loads the kg partials into the slice area and
// finishes the tile as if they were kg slices of one workgroup, so the sum
// order is fixed: slices within a workgroup, then workgroups in order.  The
// other workgroups end here.
template <typename WT, int EPI, int NMAT, int NTM, int NSS, bool COH = false>
__device__ __forceinline__ void gemm_epilogue(const GemmParams& p, int item, int M, const WaveGeo& w,
                                              f32x4 (&acc)[NTM][NMAT], const float (&ssv)[NSS], char* smem,
                                              bool has_pre = false, float2 pre = float2{0.f, 0.f}, int kgi = 0) {
    constexpr bool BF = sizeof(WT) == 2;
    constexpr bool norm = EPI != EPI_RESID;
    const int tid = tid_local(), nwaves = blockDim.x >> 6;
    const int nt = COH ? 1 : (M + 15) >> 4;             // the pass holds at most 16 rows
    const int tiles_h = p.g.ssq_tiles;
    float* rinv = (float*)smem;                              // [64]
    if (norm) {
        for (int m = w.wave; m < M; m += nwaves) {
            float s = 0.f;
            int t0 = w.lane;
            if (m == w.wave) {
#pragma unroll
                for (int u = 0; u < NSS; ++u) s += ssv[u];
                t0 = w.lane + 64 * NSS;
            }
            for (int t = t0; t < tiles_h; t += 64)
                s += COH ? poll_f32(p.SSQR + (size_t)m * tiles_h + t, p.err) : p.SSQR[(size_t)m * tiles_h + t];
#pragma unroll
            for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o);
            if (w.lane == 0) rinv[m] = 1.0f / sqrtf(s / (float)p.g.h + p.g.eps);
        }
    }
    // (every wave is past the previous epilogue's reads of the partials)
    __syncthreads();
    const int plane = nt * 16 * 16;                     // one tile's M x 16 block
    float* red = (float*)(smem + 256);                  // [tpw][ks][NMAT][plane]
    if (w.tile_ok) {
#pragma unroll
        for (int q = 0; q < NMAT; ++q)
#pragma unroll
            for (int rt = 0; rt < NTM; ++rt) {
                if (rt >= nt) break;
                float* d = red + ((size_t)(w.tl * p.ks + w.ksl) * NMAT + q) * plane;
#pragma unroll
                for (int v = 0; v < 4; ++v) d[(rt * 16 + w.grp * 4 + v) * 16 + w.j] = acc[rt][q][v];
            }
    }
    __syncthreads();
    int nsl = p.ks;                                     // slices the finish sums, in order
    if (!COH && gemm_kg(p) > 1) {
        const int kg = gemm_kg(p), n = NMAT * plane;   // one workgroup's partial (tpw = 1)
        float* mine = p.part + ((size_t)item * kg + kgi) * n;
        // only the M live rows of each matrix's 16 x 16 block travel
        for (int e = tid; e < n; e += blockDim.x) {
            if (e % plane >= M * 16) continue;
            const float* b = red + e;                   // slice sl of element e at b[sl * n]
            float v = 0.f;
            for (int sl = 0; sl < p.ks; ++sl) v += b[(size_t)sl * n];
            st_f32<true>(mine + e, v);
        }
        __builtin_amdgcn_s_waitcnt(0);                  // this thread's partials are visible device-wide
        __syncthreads();
        int* flag = (int*)red;
        if (tid == 0) {
            const unsigned old = __hip_atomic_fetch_add(p.cnt + item, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            const int lst = old + 1 == (unsigned)kg;
            if (lst) __hip_atomic_store(p.cnt + item, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            *flag = lst;
        }
        __syncthreads();
        const int lst = *flag;
        __syncthreads();
        if (!lst) return;
        const float* all = p.part + (size_t)item * kg * n;
        for (int e = tid; e < kg * n; e += blockDim.x) red[e] = e % plane < M * 16 ? ld_f32<true>(all + e) : 0.f;
        __syncthreads();
        nsl = kg;
    }
    // at most 8 k-slices in the pass (one per wave), 16 otherwise
    constexpr int KSM = COH ? 8 : 16;
    // The logits epilogue reads every element several times: its slices are
    // summed once, in place, behind one more barrier.  The other epilogues
    // sum the slices of exactly the elements each thread writes.
    constexpr bool inplace = EPI == EPI_LOGITS;
    if (inplace) {
        const int items = p.tpw * NMAT * plane;
        for (int it = tid; it < items; it += blockDim.x) {
            const int t = it / (NMAT * plane), rem = it - t * NMAT * plane;
            const int q = rem / plane, e = rem - q * plane;
            if (item * p.tpw + t >= p.tiles) continue;
            // every slice's partial is read before the sum (in slice order)
            // starts; slices past ks re-read slice 0 and add exact zeros, so
            // the loop has no branches
            float* base = red + ((size_t)(t * nsl) * NMAT + q) * plane + e;
            float part[KSM];
#pragma unroll
            for (int sl = 0; sl < KSM; ++sl) part[sl] = base[(sl < nsl ? sl : 0) * NMAT * plane];
            float sum = 0.f;
#pragma unroll
            for (int sl = 0; sl < KSM; ++sl) sum += sl < nsl ? part[sl] : 0.f;
            *base = sum;
        }
        __syncthreads();
    }
    // element (t, q, m, col): its k-slice partials summed in slice order, times
    // the row's 1/rms for the normalised kinds
    auto fin = [&](int t, int q, int m, int col) -> float {
        const float* base = red + ((size_t)(t * nsl) * NMAT + q) * plane + m * 16 + col;
        float v;
        if (inplace) {
            v = *base;
        } else {
            float part[KSM];
#pragma unroll
            for (int sl = 0; sl < KSM; ++sl) part[sl] = base[(sl < nsl ? sl : 0) * NMAT * plane];
            v = 0.f;
#pragma unroll
            for (int sl = 0; sl < KSM; ++sl) v += sl < nsl ? part[sl] : 0.f;
        }
        return norm ? v * rinv[m] : v;
    };

    if (EPI == EPI_RESID) {
        // a tile's 16 columns of one row sit in 16 consecutive lanes (blockDim
        // is a multiple of 64 and the item count a multiple of 16), so the
        // row's sum of squares over the tile is a 16-lane DPP reduction
        for (int it = tid; it < p.tpw * M * 16; it += blockDim.x) {
            const int t = it / (M * 16), rem = it - t * M * 16, m = rem >> 4, c = rem & 15;
            const int tg = item * p.tpw + t;
            if (tg >= p.tiles) continue;          // uniform over the 16 lanes of (t, m)
            const int n = tg * 16 + c;
            // residual in: Xin (row-major, written in this launch) or the row's X;
            // pre.x is this thread's first one, loaded by the caller early
            float xi;
            if (has_pre && it == tid)
                xi = pre.x;
            else if (COH && p.Xin)
                xi = poll_f32(p.Xin + (size_t)m * p.g.h + n, p.err);
            else
                xi = p.X[(size_t)p.rows[m].xrow * p.g.h + n];
            const float v = xi + fin(t, 0, m, c);
            // residual out: Xout (row-major) or the row's X
            if (COH && p.Xout)
                st_f32<true>(p.Xout + (size_t)m * p.g.h + n, f_value(v));
            else
                p.X[(size_t)p.rows[m].xrow * p.g.h + n] = v;
            const float sq = group_sum<16>(v * v);
            if (p.XBout) {
                if (BF)
                    st_u16<COH>((uint16_t*)p.XBout + (size_t)m * p.g.h + n, COH ? h_value(v) : f2h(v));
                else
                    st_f32<COH>((float*)p.XBout + (size_t)m * p.g.h + n, COH ? f_value(v) : v);
                if (c == 0) st_f32<COH>(p.SSQRout + (size_t)m * p.g.ssq_tiles + tg, COH ? f_value(sq) : sq);
            }
        }
    } else if (EPI == EPI_SWIGLU) {
        for (int it = tid; it < p.tpw * M * 16; it += blockDim.x) {
            const int t = it / (M * 16), rem = it - t * M * 16, m = rem >> 4, c = rem & 15;
            const int tg = item * p.tpw + t;
            if (tg >= p.tiles) continue;
            const float gt = fin(t, 0, m, c), up = fin(t, NMAT - 1, m, c);
            const float a = gt / (1.0f + expf(-gt)) * up;
            const size_t o = (size_t)m * p.N_mat + tg * 16 + c;
            if (BF)
                st_u16<COH>((uint16_t*)p.act + o, COH ? h_value(a) : f2h(a));
            else
                st_f32<COH>((float*)p.act + o, COH ? f_value(a) : a);
        }
    } else if (EPI == EPI_QKV) {
        const int tph = p.g.h / kTile, tpd = p.g.dh / kTile, half = p.g.dh / 2;
        for (int it = tid; it < p.tpw * M * 8; it += blockDim.x) {
            const int t = it / (M * 8), rem = it - t * M * 8, m = rem >> 3, c = rem & 7;
            const int tg = item * p.tpw + t;
            if (tg >= p.tiles) continue;
            const int mat = tg / tph, lt = tg - mat * tph, head = lt / tpd, sub = lt - head * tpd;
            const int i = sub * 8 + c;                      // pair (i, i + dh/2)
            const int pos = p.rows[m].pos;
            float x0 = fin(t, 0, m, c), x1 = fin(t, 0, m, c + 8);
            if (mat < 2) {
                // pre: this thread's first (cos, sin), loaded by the caller early
                const bool early = has_pre && it == tid;
                const float cs = early ? pre.x : p.rope[((size_t)pos * half + i) * 2];
                const float sn = early ? pre.y : p.rope[((size_t)pos * half + i) * 2 + 1];
                const float y0 = x0 * cs - x1 * sn, y1 = x1 * cs + x0 * sn;
                x0 = y0;
                x1 = y1;
            }
            const int col = head * p.g.dh + i;
            if (mat == 0) {
                st_f32<COH>(p.qout + (size_t)m * p.g.h + col, COH ? f_value(x0) : x0);
                st_f32<COH>(p.qout + (size_t)m * p.g.h + col + half, COH ? f_value(x1) : x1);
            } else {
                const int slot = p.rows[m].slot;
                const int tb = kv_table(p.g, p.stack, p.layer, p.rows[m].depth);
                const int kv = mat - 1;
                // the head's slice of the slot row, or of the committed cache
                WT* dst = slot >= 0 ? (WT*)p.kvs + kvs_index(p.g, slot, tb, kv) + head * p.g.dh
                                    : (WT*)p.kvc + kvc_index(p.g, p.rows[m].seq, tb, kv, head, pos);
                if (BF) {
                    st_u16<COH>((uint16_t*)dst + i, COH ? h_value(x0) : f2h(x0));
                    st_u16<COH>((uint16_t*)dst + i + half, COH ? h_value(x1) : f2h(x1));
                } else {
                    st_f32<COH>((float*)dst + i, COH ? f_value(x0) : x0);
                    st_f32<COH>((float*)dst + i + half, COH ? f_value(x1) : x1);
                }
            }
        }
    } else if (EPI == EPI_LOGITS) {
        for (int it = tid; it < p.tpw * M * 16; it += blockDim.x) {
            const int t = it / (M * 16), rem = it - t * M * 16, m = rem >> 4, c = rem & 15;
            const int tg = item * p.tpw + t;
            const int n = tg * 16 + c;
            if (tg >= p.tiles || n >= p.N_mat) continue;
            const float v = fin(t, 0, m, c);
            p.logits[(size_t)m * p.N_mat + n] = v;
            if (!(fabsf(v) <= 3.0e38f)) atomicOr(p.err, 1);
        }
        for (int it = tid; it < p.tpw * M; it += blockDim.x) {
            const int t = it / M, m = it - t * M;
            const int tg = item * p.tpw + t;
            if (tg >= p.tiles) continue;
            float best = -INFINITY;
            int bi = -1;
            for (int c = 0; c < 16; ++c) {
                const int n = tg * 16 + c;
                if (n >= p.N_mat) break;
                const float v = fin(t, 0, m, c);
                if (v > best || bi < 0) {
                    best = v;
                    bi = n;
                }
            }
            p.tmax[(size_t)m * p.tiles + tg] = best;
            p.targ[(size_t)m * p.tiles + tg] = bi;
        }
    }
}

// Direct path (<= 16 rows): the activation loads of the wave, the MFMAs over
// the prefetched weights, and the epilogue.  Ends with the LDS reused.
template <typename WT, int EPI, int NMAT, int MAXS, bool COH = false>
__device__ __forceinline__ void gemm_finish(const GemmParams& p, int item, int M, const BRegs<WT, NMAT, MAXS>& R,
                                            char* smem, int kgi = 0) {
    constexpr int KSTEP = WTraits<WT>::KSTEP, VEC = WTraits<WT>::VEC;
    constexpr bool norm = EPI != EPI_RESID;
    constexpr int NSS = norm ? 4 : 1;
    const WaveGeo w = wave_geo<WT, true>(p, item, kgi);
    const int tiles_h = p.g.ssq_tiles;
    // every operand load of the phase is issued before any is waited for:
    // sums of squares, the activation rows, the epilogue's first operand
    float ssv[NSS];
#pragma unroll
    for (int u = 0; u < NSS; ++u) {
        const int t = w.lane + 64 * u;
        ssv[u] = (norm && w.wave < M && t < tiles_h) ? ld_f32<COH>(p.SSQR + (size_t)w.wave * tiles_h + t) : 0.f;
    }
    // the epilogue operands of this thread's first output: RESID its residual
    // value (from Xin, row-major, when given; else the row's X), QKV the
    // (cos, sin) of its RoPE pair
    bool has_pre = false;
    float2 pre = float2{0.f, 0.f};
    const float* pre_src = nullptr;
    if (EPI == EPI_RESID) {
        const int it = tid_local();   // (opaque: the index math is redone per phase, not kept live across the pass)
        if (it < p.tpw * M * 16) {
            const int t = it / (M * 16), rem = it - t * M * 16, m = rem >> 4, c = rem & 15;
            const int tg = item * p.tpw + t;
            if (tg < p.tiles) {
                const int n = tg * 16 + c;
                if (COH && p.Xin) {
                    pre_src = p.Xin + (size_t)m * p.g.h + n;
                    pre.x = ld_f32<true>(pre_src);
                } else {
                    pre.x = p.X[(size_t)p.rows[m].xrow * p.g.h + n];
                }
                has_pre = true;
            }
        }
    } else if (EPI == EPI_QKV) {
        const int it = tid_local();   // (opaque: the index math is redone per phase, not kept live across the pass)
        if (it < p.tpw * M * 8) {
            const int t = it / (M * 8), rem = it - t * M * 8, m = rem >> 3, c = rem & 7;
            const int tg = item * p.tpw + t;
            const int tph = p.g.h / kTile, tpd = p.g.dh / kTile, half = p.g.dh / 2;
            const int mat = tg / tph, lt = tg - mat * tph, sub = (lt - (lt / tpd) * tpd);
            if (tg < p.tiles && mat < 2) {
                const float* r = p.rope + ((size_t)p.rows[m].pos * half + sub * 8 + c) * 2;
                pre = float2{r[0], r[1]};
                has_pre = true;
            }
        }
    }
    // activation rows j >= M lie beyond the resource and read as zero
    const size_t a0 = (size_t)w.s0 * KSTEP;
    const __amdgpu_buffer_rsrc_t ra =
        buf_rsrc((const WT*)(norm ? p.XB : p.abuf) + a0,
                 w.tile_ok ? (uint32_t)(((size_t)M * p.K - a0) * sizeof(WT)) : 0u);
    const int aoff = (w.j * p.K + w.grp * VEC) * (int)sizeof(WT);
    u32x4 a[MAXS];
#pragma unroll
    for (int i = 0; i < MAXS; ++i)
        a[i] = buf_load16<COH ? 16 : 0>(ra, i < w.nst ? aoff : kOutOfRange, i * KSTEP * (int)sizeof(WT));
    if (COH) {
        // fragments not yet written by their producers are read again, all of
        // them in the same round (one round trip per round)
        for (unsigned n = 0;; ++n) {
            bool miss[MAXS], any = false;
#pragma unroll
            for (int i = 0; i < MAXS; ++i) {
                miss[i] = __any(sizeof(WT) == 2 ? sentinel16(a[i]) : sentinel32(a[i]));
                any |= miss[i];
            }
            if (!any || poll_abort(n, p.err)) break;
            __builtin_amdgcn_s_sleep(1);
#pragma unroll
            for (int i = 0; i < MAXS; ++i)
                if (miss[i]) a[i] = buf_load16<16>(ra, i < w.nst ? aoff : kOutOfRange, i * KSTEP * (int)sizeof(WT));
        }
#pragma unroll
        for (int u = 0; u < NSS; ++u) {
            const int t = w.lane + 64 * u;
            if (__float_as_uint(ssv[u]) == kSentinel) ssv[u] = poll_f32(p.SSQR + (size_t)w.wave * tiles_h + t, p.err);
        }
        if (pre_src && __float_as_uint(pre.x) == kSentinel) pre.x = poll_f32(pre_src, p.err);
    }
    f32x4 acc[1][NMAT];
#pragma unroll
    for (int q = 0; q < NMAT; ++q) acc[0][q] = f32x4{0.f, 0.f, 0.f, 0.f};
    // steps past the wave's share hold zeros and add exact zeros
#pragma unroll
    for (int i = 0; i < MAXS; ++i) mfma_step<WT, NMAT>(a[i], R.b[i], acc[0]);
    gemm_epilogue<WT, EPI, NMAT, 1, NSS, COH>(p, item, M, w, acc, ssv, smem, has_pre, pre, kgi);
}

// Standalone direct path (<= 16 rows, no exchange within the launch): the
// loads are issued in an order that keeps every one of them in flight at
// once.  Vector memory loads complete in issue order, so a load issued after
// the weight stream cannot be waited for without waiting for the whole
// stream: the row descriptors the epilogue operands depend on, the RMSNorm
// partials and the activation fragments (which hit the L2) go first; then
// the weight fragments; then the epilogue's first operand, whose address
// needed the row descriptor; then the MFMAs, each waiting only for its own
// fragment.  Scheduling barriers keep the compiler from interleaving these
// groups (it would otherwise trade the loads in flight for occupancy).
template <typename WT, int EPI, int NMAT, int MAXS>
__device__ __forceinline__ void gemm_direct(const GemmParams& p, int item, int kgi, int M, char* smem) {
    constexpr int KSTEP = WTraits<WT>::KSTEP, VEC = WTraits<WT>::VEC;
    constexpr bool norm = EPI != EPI_RESID;
    constexpr int NSS = norm ? 4 : 1;
    const WaveGeo w = wave_geo<WT, true>(p, item, kgi);
    const int tiles_h = p.g.ssq_tiles;
    // (1) the row field the first epilogue operand's address needs
    const int it0 = tid_local();
    int rowf = 0, n0 = 0, sub0 = 0, m0 = 0;
    bool has_pre = false;
    if (EPI == EPI_RESID && it0 < p.tpw * M * 16) {
        const int t = it0 / (M * 16), rem = it0 - t * M * 16;
        m0 = rem >> 4;
        const int tg = item * p.tpw + t;
        if (tg < p.tiles) {
            n0 = tg * 16 + (rem & 15);
            rowf = p.rows[m0].xrow;
            has_pre = true;
        }
    } else if (EPI == EPI_QKV && it0 < p.tpw * M * 8) {
        const int t = it0 / (M * 8), rem = it0 - t * M * 8;
        m0 = rem >> 3;
        const int tg = item * p.tpw + t;
        const int tph = p.g.h / kTile, tpd = p.g.dh / kTile;
        const int mat = tg / tph, lt = tg - mat * tph;
        sub0 = (lt - (lt / tpd) * tpd) * 8 + (rem & 7);
        if (tg < p.tiles && mat < 2) {
            rowf = p.rows[m0].pos;
            has_pre = true;
        }
    }
    // (2) RMSNorm partials and activation fragments
    float ssv[NSS];
#pragma unroll
    for (int u = 0; u < NSS; ++u) {
        const int t = w.lane + 64 * u;
        ssv[u] = (norm && w.wave < M && t < tiles_h) ? p.SSQR[(size_t)w.wave * tiles_h + t] : 0.f;
    }
    const size_t a0 = (size_t)w.s0 * KSTEP;
    const __amdgpu_buffer_rsrc_t ra =
        buf_rsrc((const WT*)(norm ? p.XB : p.abuf) + a0, w.tile_ok ? (uint32_t)(((size_t)M * p.K - a0) * sizeof(WT)) : 0u);
    const int aoff = (w.j * p.K + w.grp * VEC) * (int)sizeof(WT);
    u32x4 a[MAXS];
#pragma unroll
    for (int i = 0; i < MAXS; ++i) a[i] = buf_load16<0>(ra, i < w.nst ? aoff : kOutOfRange, i * KSTEP * (int)sizeof(WT));
    __builtin_amdgcn_sched_barrier(0);
    // (3) the weight stream
    BRegs<WT, NMAT, MAXS> R;
    gemm_load_b<WT, NMAT, MAXS>(p, item, R, true, kgi);
    __builtin_amdgcn_sched_barrier(0);
    // (4) the first epilogue operand: RESID the residual value, QKV (cos, sin)
    float2 pre = float2{0.f, 0.f};
    if (has_pre) {
        if (EPI == EPI_RESID) {
            pre.x = p.X[(size_t)rowf * p.g.h + n0];
        } else {
            const float* r = p.rope + ((size_t)rowf * (p.g.dh / 2) + sub0) * 2;
            pre = float2{r[0], r[1]};
        }
    }
    __builtin_amdgcn_sched_barrier(0);
    // (5) MFMAs over the fragments in step order; steps past the wave's share
    //     hold zeros and add exact zeros
    f32x4 acc[1][NMAT];
#pragma unroll
    for (int q = 0; q < NMAT; ++q) acc[0][q] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < MAXS; ++i) mfma_step<WT, NMAT>(a[i], R.b[i], acc[0]);
    gemm_epilogue<WT, EPI, NMAT, 1, NSS, false>(p, item, M, w, acc, ssv, smem, has_pre, pre, kgi);
}

}  // namespace ls
