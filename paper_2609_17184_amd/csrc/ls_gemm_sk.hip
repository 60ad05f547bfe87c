// Stream-K weight-streaming GEMM for launches of at most 16 NT rows (NT = 1,
// 2 or 4 row tiles of 16: the decode's in-flight rows, up to 64).
//
// The packed weight matrix of a launch is one contiguous stream of 1 KB (per
// matrix) fragments, tile after tile, k step after k step (launch_pack's
// order).  A launch of G resident workgroups splits that stream into P = 4 G
// contiguous, equal ranges, one per wave: each wave streams its range in rounds
// of S k steps, double-buffered (the loads of round r+1 are in flight while
// the MFMAs of round r run), so every wave keeps loading from its first
// fragment to its last and the launch ends when the stream does, whatever
// the tile count.  A wave whose range ends a tile segment either owns the
// whole tile and runs the epilogue from its registers, or hands its partial
// (the M live rows) to the tile's first contributor without waiting, which
// sums every partial in range order (a fixed order, so results do not depend
// on timing or on how many rows share the launch) and runs the epilogue: QKV
// (RoPE on q and k, k and v written to the key/value cache of the row's own
// depth), RESID (residual add, rounded copy and per-tile sums of squares for
// the next RMSNorm), SWIGLU (silu(g) * u) or LOGITS (logits, per-tile maximum
// and its id).  The four waves of a workgroup are independent streams; their
// one barrier, at the start, publishes the rows' 1/rms (and, for wider
// launches, the rows' epilogue fields) that they compute together while their
// first round is in flight.
#include <algorithm>

#include "ls_gemm_dev.h"

namespace ls {

constexpr int kSkWaves = 4;
constexpr int kSkMinSteps = 32;        // k steps per wave at least (16-row launches)
constexpr int kSkMinStepsWide = 32;    // (launches of 32 or 64 rows)

__device__ __forceinline__ long long sk_wave_of(long long u, long long P, long long U) {
    return ((u + 1) * P - 1) / U;     // the wave whose range [U w / P, U (w+1) / P) holds unit u
}

// A wave-uniform value the compiler may have computed in vector registers,
// moved to scalar ones (so buffer resources built from it need no waterfall loop)
__device__ __forceinline__ const void* sk_uniform(const void* p) {
    const uint64_t v = (uint64_t)p;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return (const void*)(((uint64_t)hi << 32) | lo);
}

template <typename WT, int NMAT, int S, int NT>
__device__ __forceinline__ void sk_load(const GemmParams& p, int ns, long long u, int n, int lane, int M, int ntl,
                                        u32x4 (&B)[S][NMAT], u32x4 (&A)[S][NT]) {
    constexpr int KSTEP = WTraits<WT>::KSTEP, VEC = WTraits<WT>::VEC;
    const int s = (int)(u % ns);
    // (n = 0: an empty range at any base, every load returns zeros)
    const __amdgpu_buffer_rsrc_t rb =
        buf_rsrc(sk_uniform((const char*)p.Wp + (n ? (size_t)u * NMAT * 1024 : 0)),
                 __builtin_amdgcn_readfirstlane((uint32_t)n * NMAT * 1024));
    const int vb = lane * 16;
#pragma unroll
    for (int i = 0; i < S; ++i)
#pragma unroll
        for (int q = 0; q < NMAT; ++q) B[i][q] = buf_load16<2>(rb, i < n ? vb : kOutOfRange, (i * NMAT + q) * 1024);
    // activation fragments of the same steps, 16 rows per row tile (rows >= M
    // lie beyond the range: zeros; row tiles past the live ones are not read)
    const WT* a0 = (const WT*)p.abuf + (size_t)s * KSTEP;
    const __amdgpu_buffer_rsrc_t ra =
        buf_rsrc(sk_uniform(a0),
                 __builtin_amdgcn_readfirstlane(n ? (uint32_t)(((size_t)M * p.K - (size_t)s * KSTEP) * sizeof(WT)) : 0u));
    const int va = ((lane & 15) * p.K + (lane >> 4) * VEC) * (int)sizeof(WT);
    const int rstride = 16 * p.K * (int)sizeof(WT);
#pragma unroll
    for (int i = 0; i < S; ++i)
#pragma unroll
        for (int rt = 0; rt < NT; ++rt)
            A[i][rt] = buf_load16<0>(ra, (i < n && rt < ntl) ? va + rt * rstride : kOutOfRange,
                                     i * KSTEP * (int)sizeof(WT));
}

// 1/rms of rows 0..M-1 into r[0..M) (workgroup LDS), from the per-tile sums
// of squares: wave wv takes rows wv, wv + 4, ..., 16 lanes per row, four rows
// per pass (the caller's barrier publishes them)
__device__ __forceinline__ void sk_rinv(const GemmParams& p, int M, int wv, int lane, float* r) {
    const int T = p.g.ssq_tiles, sub = lane & 15;
    for (int m0 = wv; m0 < M; m0 += 4 * kSkWaves) {
        const int m = m0 + (lane >> 4) * kSkWaves;
        float s = 0.f;
        if (m < M) {
            const float* src = p.SSQR + (size_t)m * T;
#pragma unroll 8
            for (int t = sub; t < T; t += 16) s += src[t];
        }
        s = group_sum<16>(s);
        if (sub == 0 && m < M) r[m] = 1.0f / sqrtf(s / (float)p.g.h + p.g.eps);
    }
}

// The row fields an epilogue reads, copied to LDS once per workgroup
struct SkRowMeta {
    int xrow, pos, slot, seq, depth;
};

// Epilogue operands of tile t loaded ahead of its finish: RESID the residual
// values of the lane's rows, QKV the (cos, sin) of its RoPE pair per row.
template <int NT>
struct SkPre {
    int t;                 // tile they belong to (-1: none)
    f32x4 a[NT], b[NT];
};

// (meta: the rows' fields in LDS, else null: read from the row list)
template <int EPI, int NT>
__device__ __forceinline__ SkPre<NT> sk_prefetch(const GemmParams& p, int t, int M, int lane,
                                                 const SkRowMeta* meta = nullptr) {
    SkPre<NT> r;
    r.t = t;
    const int j = lane & 15, grp = lane >> 4;
#pragma unroll
    for (int rt = 0; rt < NT; ++rt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            r.a[rt][v] = 0.f;
            r.b[rt][v] = 0.f;
        }
    if (EPI == EPI_RESID) {
#pragma unroll
        for (int rt = 0; rt < NT; ++rt)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int m = rt * 16 + grp * 4 + v;
                if (m < M) r.a[rt][v] = p.X[(size_t)(meta ? meta[m].xrow : p.rows[m].xrow) * p.g.h + t * 16 + j];
            }
    } else if (EPI == EPI_QKV) {
        const int tph = p.g.h / kTile, tpd = p.g.dh / kTile, half = p.g.dh / 2;
        const int mat = t / tph, lt = t - mat * tph, sub = lt - (lt / tpd) * tpd;
        if (mat < 2 && j < 8) {
#pragma unroll
            for (int rt = 0; rt < NT; ++rt)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int m = rt * 16 + grp * 4 + v;
                    if (m < M) {
                        const int pos = meta ? meta[m].pos : p.rows[m].pos;
                        const float* rp = p.rope + ((size_t)pos * half + sub * 8 + j) * 2;
                        r.a[rt][v] = rp[0];
                        r.b[rt][v] = rp[1];
                    }
                }
        }
    }
    return r;
}

// Epilogue of tile t over rows r0 .. r0+15 from the wave's summed
// accumulators: lane l holds rows r0 + 4 (l / 16) + v (v = 0..3) of column
// l % 16 of each matrix.  have: pa / pb hold the prefetched operands.
template <typename WT, int EPI, int NMAT>
__device__ __forceinline__ void sk_finish(const GemmParams& p, int t, int M, int r0, int lane,
                                          const f32x4 (&acc)[NMAT], const float* rinv, const SkRowMeta* meta,
                                          bool have, f32x4 pa, f32x4 pb) {
    constexpr bool BF = sizeof(WT) == 2;
    const int j = lane & 15, grp = lane >> 4;
    // every load of the epilogue is issued before its first store (the stores
    // may alias them as far as the compiler knows, which would serialise them)
    if (EPI == EPI_RESID) {
        const int n = t * 16 + j;
        int xr[4];
        float xin[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int m = r0 + grp * 4 + v;
            xr[v] = m < M ? (meta ? meta[m].xrow : p.rows[m].xrow) : 0;
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int m = r0 + grp * 4 + v;
            xin[v] = have ? pa[v] : m < M ? p.X[(size_t)xr[v] * p.g.h + n] : 0.f;
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int m = r0 + grp * 4 + v;
            float out = 0.f;
            if (m < M) {
                out = xin[v] + acc[0][v];
                p.X[(size_t)xr[v] * p.g.h + n] = out;
            }
            const float sq = group_sum<16>(out * out);
            if (m < M && p.XBout) {
                if (BF)
                    ((uint16_t*)p.XBout)[(size_t)m * p.g.h + n] = f2h(out);
                else
                    ((float*)p.XBout)[(size_t)m * p.g.h + n] = out;
                if (j == 0) p.SSQRout[(size_t)m * p.g.ssq_tiles + t] = sq;
            }
        }
    } else if (EPI == EPI_SWIGLU) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int m = r0 + grp * 4 + v;
            if (m >= M) continue;
            const float r = rinv[m];
            const float gt = acc[0][v] * r, up = acc[NMAT - 1][v] * r;
            const float a = gt / (1.0f + expf(-gt)) * up;
            const size_t o = (size_t)m * p.N_mat + t * 16 + j;
            if (BF)
                ((uint16_t*)p.act)[o] = f2h(a);
            else
                ((float*)p.act)[o] = a;
        }
    } else if (EPI == EPI_QKV) {
        const int tph = p.g.h / kTile, tpd = p.g.dh / kTile, half = p.g.dh / 2;
        const int mat = t / tph, lt = t - mat * tph, head = lt / tpd, sub = lt - head * tpd;
        const int i = sub * 8 + (j & 7);                  // pair (i, i + dh/2)
        int pos[4], slot[4], seq[4], dep[4];
        float cs[4], sn[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int m = r0 + grp * 4 + v;
            pos[v] = slot[v] = seq[v] = dep[v] = 0;
            if (m < M) {
                if (meta) {
                    const SkRowMeta& r = meta[m];
                    pos[v] = r.pos;
                    if (mat > 0) {
                        slot[v] = r.slot;
                        seq[v] = r.seq;
                        dep[v] = r.depth;
                    }
                } else {
                    const Row& r = p.rows[m];
                    pos[v] = r.pos;
                    if (mat > 0) {
                        slot[v] = r.slot;
                        seq[v] = r.seq;
                        dep[v] = r.depth;
                    }
                }
            }
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int m = r0 + grp * 4 + v;
            cs[v] = pa[v];
            sn[v] = pb[v];
            if (!have && mat < 2 && j < 8 && m < M) {
                cs[v] = p.rope[((size_t)pos[v] * half + i) * 2];
                sn[v] = p.rope[((size_t)pos[v] * half + i) * 2 + 1];
            }
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int m = r0 + grp * 4 + v;
            const float x = m < M ? acc[0][v] * rinv[m] : 0.f;
            const float partner = __shfl_xor(x, 8);      // column j + 8 holds the pair's second half
            if (m >= M || j >= 8) continue;
            float x0 = x, x1 = partner;
            if (mat < 2) {
                const float y0 = x0 * cs[v] - x1 * sn[v], y1 = x1 * cs[v] + x0 * sn[v];
                x0 = y0;
                x1 = y1;
            }
            const int col = head * p.g.dh + i;
            if (mat == 0) {
                p.qout[(size_t)m * p.g.h + col] = x0;
                p.qout[(size_t)m * p.g.h + col + half] = x1;
            } else {
                const int tb = kv_table(p.g, p.stack, p.layer, dep[v]);
                WT* dst = slot[v] >= 0 ? (WT*)p.kvs + kvs_index(p.g, slot[v], tb, mat - 1) + head * p.g.dh
                                       : (WT*)p.kvc + kvc_index(p.g, seq[v], tb, mat - 1, head, pos[v]);
                if (BF) {
                    ((uint16_t*)dst)[i] = f2h(x0);
                    ((uint16_t*)dst)[i + half] = f2h(x1);
                } else {
                    ((float*)dst)[i] = x0;
                    ((float*)dst)[i + half] = x1;
                }
            }
        }
    } else if (EPI == EPI_LOGITS) {
        const int n = t * 16 + j;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int m = r0 + grp * 4 + v;
            const bool live = m < M && n < p.N_mat;
            const float val = live ? acc[0][v] * rinv[m] : 0.f;
            if (live) {
                p.logits[(size_t)m * p.N_mat + n] = val;
                if (!(fabsf(val) <= 3.0e38f)) atomicOr(p.err, 1);
            }
            // the tile's maximum over its 16 columns, ties to the lowest id
            float bv = live ? val : -INFINITY;
            int bi = live ? n : -1;
#pragma unroll
            for (int o = 8; o >= 1; o >>= 1) {
                const float ov = __shfl_xor(bv, o);
                const int oi = __shfl_xor(bi, o);
                if (oi >= 0 && (bi < 0 || ov > bv || (ov == bv && oi < bi))) {
                    bv = ov;
                    bi = oi;
                }
            }
            if (m < M && j == 0) {
                p.tmax[(size_t)m * p.tiles + t] = bv;
                p.targ[(size_t)m * p.tiles + t] = bi;
            }
        }
    }
}

template <typename WT, int EPI, int NMAT, int S, int NT>
__global__ void __launch_bounds__(kSkWaves * 64) __attribute__((amdgpu_waves_per_eu(NT == 1 ? 1 : 2))) k_gemm_sk(GemmParams p) {
    __shared__ float rinv[16 * NT];
    __shared__ SkRowMeta meta[16 * NT];
    const int M = min(ld_uniform(p.nrows), 16 * NT);       // (the host sizes NT from the row capacity)
    if (M <= 0) return;
    // the wave index is wave-uniform: the stream geometry and the buffer
    // resources derived from it stay in scalar registers
    const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int ntl = NT == 1 ? 1 : (M + 15) / 16;           // live row tiles (M <= 16 NT)
    constexpr int KSTEP = WTraits<WT>::KSTEP;
    GemmParams q = p;
    if (EPI != EPI_RESID) q.abuf = p.XB;                   // the A operand of the normalised kinds
    const int ns = p.K / KSTEP;
    const long long U = (long long)p.tiles * ns, P = (long long)gridDim.x * kSkWaves;
    const long long w = (long long)blockIdx.x * kSkWaves + wv;
    const long long u0 = U * w / P, u1 = U * (w + 1) / P;
    auto round_len = [&](long long u) -> int {
        const long long r = min((long long)S, min(u1 - u, (long long)ns - u % ns));
        return (int)r;
    };
    f32x4 acc[NT][NMAT];
#pragma unroll
    for (int rt = 0; rt < NT; ++rt)
#pragma unroll
        for (int k = 0; k < NMAT; ++k) acc[rt][k] = f32x4{0.f, 0.f, 0.f, 0.f};
    // the tile this wave may finish at the end of the launch (its last
    // segment's tile: every other contributor of it ends earlier or at the same
    // time) has its epilogue operands loaded now (16-row launches: wider ones
    // have no registers to hold them through the stream)
    const SkPre<NT> pre = NT == 1 && u0 < u1 ? sk_prefetch<EPI, NT>(q, (int)((u1 - 1) / ns), M, lane) : SkPre<NT>{-1, {}, {}};
    auto finish = [&](int t, const f32x4 (&a)[NT][NMAT]) __attribute__((always_inline)) {
        if (NT > 1 && (EPI == EPI_RESID || EPI == EPI_QKV)) {
            // the epilogue operands of every row tile in one round trip
            const SkPre<NT> g = sk_prefetch<EPI, NT>(q, t, M, lane, meta);
#pragma unroll
            for (int rt = 0; rt < NT; ++rt)
                if (rt < ntl) sk_finish<WT, EPI, NMAT>(q, t, M, rt * 16, lane, a[rt], rinv, meta, true, g.a[rt], g.b[rt]);
        } else {
#pragma unroll
            for (int rt = 0; rt < NT; ++rt)
                if (rt < ntl)
                    sk_finish<WT, EPI, NMAT>(q, t, M, rt * 16, lane, a[rt], rinv, NT > 1 ? meta : nullptr, pre.t == t,
                                             pre.a[rt], pre.b[rt]);
        }
    };
    // the end of a tile segment: finish the tile, or hand the partial to the
    // tile's first contributor.  A tile shared by several waves is finished by
    // the wave holding its first k steps: they end that wave's range, so it
    // reaches them last (the other contributors hold the tile's later steps at
    // the start of their ranges, or all of their ranges).  The others store
    // their partials and stream on without waiting; the partial slots hold the
    // sentinel between launches, and the finishing wave reads each partial
    // once it holds no sentinel, adds them in range order and clears the slots.
    auto flush = [&](long long u_end) __attribute__((always_inline)) {
        const int t = (int)((u_end - 1) / ns);
        const long long a = (long long)t * ns, b = a + ns;
        const int wlo = (int)sk_wave_of(a, P, U), nct = (int)sk_wave_of(b - 1, P, U) - wlo + 1;
        if (nct > 1) {
            const int k = (int)w - wlo, grp = lane >> 4, jj = lane & 15;
            float* all = p.part + (size_t)t * p.kg * NT * NMAT * 256;
            if (k != 0) {
                float* part = all + (size_t)k * NT * NMAT * 256;
#pragma unroll
                for (int rt = 0; rt < NT; ++rt)
#pragma unroll
                    for (int m = 0; m < NMAT; ++m)
#pragma unroll
                        for (int v = 0; v < 4; ++v)
                            if (rt * 16 + grp * 4 + v < M)
                                st_f32<true>(part + (rt * NMAT + m) * 256 + (grp * 4 + v) * 16 + jj, f_value(acc[rt][m][v]));
                return;
            }
            // the other partials added to the wave's own, CB contributors at a time (one round trip per
            // CB, repeated while a slot still holds the sentinel; CB keeps the
            // kernel's registers within its occupancy)
            constexpr int CB = NT == 1 ? 2 : 1;
            for (int c0 = 1; c0 < nct; c0 += CB) {
                float x[CB][NT][NMAT][4];
                for (unsigned n = 0;; ++n) {
                    bool miss = false;
#pragma unroll
                    for (int cc = 0; cc < CB; ++cc)
#pragma unroll
                        for (int rt = 0; rt < NT; ++rt)
#pragma unroll
                            for (int m = 0; m < NMAT; ++m)
#pragma unroll
                                for (int v = 0; v < 4; ++v) {
                                    const int c = c0 + cc;
                                    const bool live = c < nct && rt * 16 + grp * 4 + v < M;
                                    x[cc][rt][m][v] =
                                        live ? ld_f32<true>(all + (((size_t)c * NT + rt) * NMAT + m) * 256 + (grp * 4 + v) * 16 + jj)
                                             : 0.f;
                                    miss |= live && __float_as_uint(x[cc][rt][m][v]) == kSentinel;
                                }
                    if (!__ballot(miss) || poll_abort(n, p.err)) break;
                    __builtin_amdgcn_s_sleep(1);
                }
#pragma unroll
                for (int cc = 0; cc < CB; ++cc) {
                    const int c = c0 + cc;
                    if (c >= nct) break;
#pragma unroll
                    for (int rt = 0; rt < NT; ++rt)
#pragma unroll
                        for (int m = 0; m < NMAT; ++m)
#pragma unroll
                            for (int v = 0; v < 4; ++v) {
                                acc[rt][m][v] += x[cc][rt][m][v];
                                if (rt * 16 + grp * 4 + v < M)
                                    st_f32<true>(all + (((size_t)c * NT + rt) * NMAT + m) * 256 + (grp * 4 + v) * 16 + jj,
                                                 __uint_as_float(kSentinel));
                            }
                }
            }
        }
        finish(t, acc);
    };
    u32x4 B0[S][NMAT], B1[S][NMAT], A0[S][NT], A1[S][NT];
    long long u = u0;
    int n0 = u < u1 ? round_len(u) : 0, n1 = 0;
    auto mfma_round = [&](const u32x4 (&A)[S][NT], const u32x4 (&B)[S][NMAT]) {
#pragma unroll
        for (int i = 0; i < S; ++i)
#pragma unroll
            for (int rt = 0; rt < NT; ++rt)
                if (rt < ntl) mfma_step<WT, NMAT>(A[i][rt], B[i], acc[rt]);
    };
    auto clear = [&]() {
#pragma unroll
        for (int rt = 0; rt < NT; ++rt)
#pragma unroll
            for (int k = 0; k < NMAT; ++k) acc[rt][k] = f32x4{0.f, 0.f, 0.f, 0.f};
    };
    if (n0) sk_load<WT, NMAT, S, NT>(q, ns, u, n0, lane, M, ntl, B0, A0);
    // 1/rms of the rows and (launches of more than 16 rows) the rows'
    // epilogue fields, shared by the workgroup's waves, while the first round
    // is in flight (every wave reaches this barrier once)
    if (EPI != EPI_RESID) sk_rinv(p, M, wv, lane, rinv);
    if (NT > 1 && (EPI == EPI_RESID || EPI == EPI_QKV))
        for (int m = threadIdx.x; m < M; m += kSkWaves * 64) {
            const Row& r = p.rows[m];
            meta[m] = SkRowMeta{r.xrow, r.pos, r.slot, r.seq, r.depth};
        }
    __syncthreads();
    while (n0) {
        // ---- round in B0 / A0 ------------------------------------------------
        long long un = u + n0;
        n1 = un < u1 ? round_len(un) : 0;
        // issued even when no round follows (zeros from an empty range): the
        // MFMAs below then wait for exactly the loads issued before these, so
        // the next round stays in flight while they run
        sk_load<WT, NMAT, S, NT>(q, ns, un, n1, lane, M, ntl, B1, A1);
        mfma_round(A0, B0);
        if (un % ns == 0 || un == u1) {
            flush(un);
            clear();
        }
        if (!n1) break;
        u = un;
        // ---- round in B1 / A1 ------------------------------------------------
        un = u + n1;
        n0 = un < u1 ? round_len(un) : 0;
        sk_load<WT, NMAT, S, NT>(q, ns, un, n0, lane, M, ntl, B0, A0);
        mfma_round(A1, B1);
        if (un % ns == 0 || un == u1) {
            flush(un);
            clear();
        }
        u = un;
    }
}

// k steps per round.  16 rows: one workgroup per CU, so one wave per SIMD,
// each with two rounds in flight (6 k steps of two matrices or 9 of one: 12
// or 9 KB per round; measured against 4–18).  With several waves per SIMD the
// arbiter serves the oldest first, so the waves of the workgroups placed
// first on a CU end their (equal) ranges long before the last ones, and the
// launch's tail runs on a fraction of the CU's requests; a single wave per
// SIMD has no such skew.  32 and 64 rows: one workgroup per CU too, with
// rounds sized for two waves per SIMD (the NT activation fragments per step
// take the registers; the 64-row residual variant also holds its epilogue
// operands of four row tiles).
template <int EPI, int NMAT, int NT>
constexpr int sk_steps() {
    return NT == 1 ? (NMAT == 2 ? 6 : 9) : EPI == EPI_RESID && NT == 4 ? 2 : 16 / (NMAT + NT);
}

template <typename WT, int EPI, int NMAT>
static const void* sk_fn(int nt) {
    switch (nt) {
        case 1: return (const void*)k_gemm_sk<WT, EPI, NMAT, sk_steps<EPI, NMAT, 1>(), 1>;
        case 2: return (const void*)k_gemm_sk<WT, EPI, NMAT, sk_steps<EPI, NMAT, 2>(), 2>;
        case 4: return (const void*)k_gemm_sk<WT, EPI, NMAT, sk_steps<EPI, NMAT, 4>(), 4>;
    }
    return nullptr;
}

static const void* sk_kernel(int epi, bool bf16, int nt) {
    if (bf16) {
        switch (epi) {
            case EPI_QKV: return sk_fn<uint16_t, EPI_QKV, 1>(nt);
            case EPI_RESID: return sk_fn<uint16_t, EPI_RESID, 1>(nt);
            case EPI_SWIGLU: return sk_fn<uint16_t, EPI_SWIGLU, 2>(nt);
            case EPI_LOGITS: return sk_fn<uint16_t, EPI_LOGITS, 1>(nt);
        }
    } else {
        switch (epi) {
            case EPI_QKV: return sk_fn<float, EPI_QKV, 1>(nt);
            case EPI_RESID: return sk_fn<float, EPI_RESID, 1>(nt);
            case EPI_SWIGLU: return sk_fn<float, EPI_SWIGLU, 2>(nt);
            case EPI_LOGITS: return sk_fn<float, EPI_LOGITS, 1>(nt);
        }
    }
    return nullptr;
}

// Launch shape of a stream-K GEMM: every workgroup resident at once, and at
// least one k step per wave.  *grid = 0 when the launch has fewer k steps
// than a workgroup has waves (the tiled direct path runs it instead).
// *contrib: the most waves a tile's stream can be split over (partial slots).
hipError_t gemm_sk_shape(int epi, bool bf16, int nt, int tiles, int K, int* grid, int* contrib) {
    *grid = 0;
    *contrib = 0;
    const void* f = sk_kernel(epi, bf16, nt);
    if (!f) return hipErrorInvalidValue;
    int dev = 0, cus = 0, per = 0;
    hipError_t e;
    if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
    if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, f, kSkWaves * 64, 0)) != hipSuccess) return e;
    per = std::min(per, 1);   // one workgroup per CU: no SIMD holds waves of two workgroups (see sk_steps)
    const long long ns = K / (bf16 ? 32 : 16), U = (long long)tiles * ns;
    // every workgroup resident, and at least kSkMinSteps k steps per wave (a
    // shorter share spends more on its tile's fix-up than on its stream)
    long long G = (long long)cus * std::max(per, 1);
    G = std::min(G, U / (kSkWaves * (nt == 1 ? kSkMinSteps : kSkMinStepsWide)));
    if (G < 1) G = U / kSkWaves;
    if (G < 1) return hipSuccess;          // too few k steps to give every wave one: not used
    const long long P = G * kSkWaves, minw = U / P;
    *grid = (int)G;
    *contrib = (int)((ns + minw - 1) / minw + 1);
    return hipSuccess;
}

hipError_t launch_gemm_sk(const GemmParams& p, int epi, bool bf16, int nt, int grid, hipStream_t st) {
    const void* f = sk_kernel(epi, bf16, nt);
    if (!f || grid < 1) return hipErrorInvalidValue;
    GemmParams q = p;
    void* args[] = {(void*)&q};
    return ls_launch(f, dim3(grid), dim3(kSkWaves * 64), args, 0, st);
}

}  // namespace ls
