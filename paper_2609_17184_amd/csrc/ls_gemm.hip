// Weight-streaming skinny GEMM for the batched recurrent step, with the
// block's RMSNorm and pointwise work fused in.
//
// One decode step of LoopSpec advances every active branch by one recurrent
// depth in a single batched call to the shared blocks (Sec. 4.2, "Batched
// Recurrence"); the branches sit at different depths but share one pass over
// the weights.  With M <= 64 rows the work is an HBM-bound stream of the
// weight matrix: out[m][n] = sum_k A[m][k] * W[n][k].
//
// Layout of the computation
//   * a tile is 16 output features (one MFMA 16x16 B operand); a workgroup
//     holds `tpw` tiles x `ks` k-slices, one wavefront each;
//   * k is cut in steps of one 16-byte load per lane (32 bf16 or 16 fp32
//     values of a row); wave (tile, slice) owns the steps s with s % ks == slice
//     and accumulates them in increasing s; the slices are summed in slice
//     order at the end.  The arithmetic depends only on (K, ks), never on the
//     number of rows or on a row's position: every row's result is
//     bit-identical however many branches share the pass;
//   * RMSNorm: A is the hidden state rounded to the weight dtype, the norm
//     gain is folded into the weights (W'[n][k] = W[n][k] g[k]) and the row's
//     1/rms multiplies the result: out = rinv[m] * sum_k xb[m][k] W'[n][k];
//   * decode launches (<= 16 rows): every lane issues all its 16-byte weight
//     loads (nontemporal: streamed once per step) and its A loads at entry and
//     feeds v_mfma_f32_16x16x32_bf16 from registers -- one memory round trip,
//     no LDS staging; larger launches (prefill, 64 rows) stage A through LDS;
//   * epilogues: QKV (RoPE on q and k, K/V written to the KV cache of the
//     row's own depth), RESID (residual add, rounded copy and per-16-column
//     sums of squares for the next RMSNorm), SWIGLU (silu(g) * u), LOGITS
//     (logits + per-tile max / arg-max for the vocabulary-sharded readout).
#include "ls_gemm.h"

#include <algorithm>

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
__device__ __forceinline__ int tile_row(const GemmParams& p, int tile, int j, int* mat) {
    if (EPI == EPI_QKV) {
        const int tph = p.g.h / kTile;              // tiles per matrix
        const int m = tile / tph, lt = tile - m * tph;
        const int tpd = p.g.dh / kTile;             // tiles per head
        const int head = lt / tpd, sub = lt - head * tpd;
        // columns j and j+8 hold a RoPE pair (i, i + dh/2)
        const int c = j < 8 ? sub * 8 + j : p.g.dh / 2 + sub * 8 + (j - 8);
        *mat = m;
        return head * p.g.dh + c;
    }
    *mat = 0;
    return tile * kTile + j;
}

template <typename WT, int NMAT>
__device__ __forceinline__ void mfma_step(const u32x4& a, const u32x4 (&b)[NMAT], f32x4 (&acc)[NMAT]) {
    if (sizeof(WT) == 2) {
        const bf16x8 av = __builtin_bit_cast(bf16x8, a);
#pragma unroll
        for (int q = 0; q < NMAT; ++q)
            acc[q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, __builtin_bit_cast(bf16x8, b[q]), acc[q], 0, 0, 0);
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

template <typename WT, int EPI, int NMAT, int NTM>
__global__ void __launch_bounds__(1024) k_gemm(GemmParams p) {
    using T = WTraits<WT>;
    constexpr int KSTEP = T::KSTEP;
    constexpr int VEC = T::VEC;
    constexpr int MAXS = gemm_max_steps(EPI, NTM);
    constexpr bool BF = sizeof(WT) == 2;
    constexpr bool norm = EPI != EPI_RESID;        // A is the RMS-normalised hidden state

    extern __shared__ __align__(16) char smem[];
    const int M = *p.nrows;
    if (M <= 0) return;
    const int nt = (M + 15) >> 4;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int nwaves = blockDim.x >> 6;
    const int tl = wave / p.ks, ksl = wave - tl * p.ks;
    const int tile = blockIdx.x * p.tpw + tl;
    const bool tile_ok = tile < p.tiles;
    const int j = lane & 15, grp = lane >> 4;
    const int nsteps = p.K / KSTEP;
    // k steps of this wave: a contiguous block (direct path) or every ks-th step
    // (LDS path, where all waves consume the same staged chunk together)
    const int s0 = NTM == 1 ? (int)(((long)nsteps * ksl) / p.ks) : 0;
    const int nst = NTM == 1 ? (int)(((long)nsteps * (ksl + 1)) / p.ks) - s0
                             : (ksl < nsteps ? (nsteps - ksl + p.ks - 1) / p.ks : 0);
    const WT* Abase = (const WT*)(norm ? p.XB : p.abuf);

    float* rinv = (float*)smem;                              // [64]

    // ---- RMSNorm statistics of row `wave`: loads issued first, used last ----
    constexpr int NSS = norm ? 4 : 1;
    float ssv[NSS];
    const int tiles_h = p.g.ssq_tiles;
#pragma unroll
    for (int u = 0; u < NSS; ++u) {
        const int t = lane + 64 * u;
        ssv[u] = (norm && wave < M && t < tiles_h) ? p.SSQR[(size_t)wave * tiles_h + t] : 0.f;
    }

    // ---- packed B: this tile's blocks, lane offset applied ------------------
    const WT* bt = (const WT*)p.Wp + (size_t)(tile_ok ? tile : 0) * nsteps * NMAT * 64 * VEC + lane * VEC;
    const bool bvalid = tile_ok;

    f32x4 acc[NTM][NMAT];
#pragma unroll
    for (int rt = 0; rt < NTM; ++rt)
#pragma unroll
        for (int q = 0; q < NMAT; ++q) acc[rt][q] = f32x4{0.f, 0.f, 0.f, 0.f};

    if constexpr (NTM == 1) {
        // ---- direct operands: A (rows j < M) and W, all loads issued at entry ----
        // this wave owns the contiguous steps [s0, s0 + nst) of the tile
        const WT* arow = Abase + (size_t)j * p.K + grp * VEC;
        const bool aval = j < M && tile_ok;
        for (int i0 = 0; i0 < nst; i0 += MAXS) {
            u32x4 a[MAXS];
            u32x4 b[MAXS][NMAT];
#pragma unroll
            for (int i = 0; i < MAXS; ++i) {
                const int s = s0 + i0 + i;
                a[i] = (i0 + i < nst && aval) ? *(const u32x4*)(arow + (size_t)s * KSTEP) : u32x4{0u, 0u, 0u, 0u};
            }
#pragma unroll
            for (int i = 0; i < MAXS; ++i) {
                const int s = s0 + i0 + i;
#pragma unroll
                for (int q = 0; q < NMAT; ++q)
                    b[i][q] = (i0 + i < nst && bvalid)
                                  ? __builtin_nontemporal_load(
                                        (const u32x4*)(bt + ((size_t)s * NMAT + q) * 64 * VEC))
                                  : u32x4{0u, 0u, 0u, 0u};
            }
#pragma unroll
            for (int i = 0; i < MAXS; ++i)
                if (i0 + i < nst) mfma_step<WT, NMAT>(a[i], b[i], acc[0]);
        }
    } else {
        // ---- A staged through LDS (up to 64 rows), weights in rounds of MAXS ----
        WT* A = (WT*)(smem + 256);                           // [nt*16][astride]
        const int astride = p.kc + VEC;                      // 16-byte row pad
        const int span = MAXS * p.ks;
        for (int r0 = 0; r0 < nsteps; r0 += span) {
            const int ibase = r0 / p.ks;
            u32x4 b[MAXS][NMAT];
#pragma unroll
            for (int i = 0; i < MAXS; ++i) {
                const int s = ksl + (ibase + i) * p.ks;
#pragma unroll
                for (int q = 0; q < NMAT; ++q)
                    b[i][q] = (ibase + i < nst && bvalid)
                                  ? __builtin_nontemporal_load(
                                        (const u32x4*)(bt + ((size_t)s * NMAT + q) * 64 * VEC))
                                  : u32x4{0u, 0u, 0u, 0u};
            }
            const int kend = min(p.K, (r0 + span) * KSTEP);
            for (int c0 = r0 * KSTEP; c0 < kend; c0 += p.kc) {
                const int kc = min(p.kc, kend - c0);
                __syncthreads();
                const int vpr = kc / VEC;
                for (int it = tid; it < nt * 16 * vpr; it += blockDim.x) {
                    const int m = it / vpr, kv = (it - m * vpr) * VEC;
                    *(u32x4*)(A + m * astride + kv) =
                        m < M ? *(const u32x4*)(Abase + (size_t)m * p.K + c0 + kv) : u32x4{0u, 0u, 0u, 0u};
                }
                __syncthreads();
                if (!tile_ok) continue;
                const int s_lo = c0 / KSTEP, s_hi = (c0 + kc) / KSTEP;
#pragma unroll
                for (int i = 0; i < MAXS; ++i) {
                    const int ss = ksl + (ibase + i) * p.ks;
                    if (ibase + i >= nst || ss < s_lo || ss >= s_hi) continue;
                    const int ko = (ss - s_lo) * KSTEP + grp * VEC;
#pragma unroll
                    for (int rt = 0; rt < NTM; ++rt) {
                        if (rt >= nt) break;
                        const u32x4 a = *(const u32x4*)(A + (rt * 16 + j) * astride + ko);
                        mfma_step<WT, NMAT>(a, b[i], acc[rt]);
                    }
                }
            }
        }
    }

    // ---- 1/rms of each row ----------------------------------------------------
    if (norm) {
        for (int m = wave; m < M; m += nwaves) {
            float s = 0.f;
            int t0 = lane;
            if (m == wave) {
#pragma unroll
                for (int u = 0; u < NSS; ++u) s += ssv[u];
                t0 = lane + 64 * NSS;
            }
            for (int t = t0; t < tiles_h; t += 64) s += p.SSQR[(size_t)m * tiles_h + t];
#pragma unroll
            for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o);
            if (lane == 0) rinv[m] = 1.0f / sqrtf(s / (float)p.g.h + p.g.eps);
        }
    }

    // ---- cross-wave reduction in slice order --------------------------------
    __syncthreads();
    const int plane = nt * 16 * 16;                     // one tile's M x 16 block
    float* red = (float*)(smem + 256);                  // [tpw][ks][NMAT][plane]
    if (tile_ok) {
#pragma unroll
        for (int q = 0; q < NMAT; ++q)
#pragma unroll
            for (int rt = 0; rt < NTM; ++rt) {
                if (rt >= nt) break;
                float* d = red + ((size_t)(tl * p.ks + ksl) * NMAT + q) * plane;
#pragma unroll
                for (int v = 0; v < 4; ++v) d[(rt * 16 + grp * 4 + v) * 16 + j] = acc[rt][q][v];
            }
    }
    __syncthreads();
    {
        const int items = p.tpw * NMAT * plane;
        for (int it = tid; it < items; it += blockDim.x) {
            const int t = it / (NMAT * plane), rem = it - t * NMAT * plane;
            const int q = rem / plane, e = rem - q * plane;
            if (blockIdx.x * p.tpw + t >= p.tiles) continue;
            float sum = 0.f;
            for (int sl = 0; sl < p.ks; ++sl) sum += red[((size_t)(t * p.ks + sl) * NMAT + q) * plane + e];
            red[((size_t)(t * p.ks) * NMAT + q) * plane + e] = sum;
        }
    }
    __syncthreads();
    auto fin = [&](int t, int q, int m, int col) -> float {
        const float v = red[((size_t)(t * p.ks) * NMAT + q) * plane + m * 16 + col];
        return norm ? v * rinv[m] : v;
    };

    // ---- epilogues ----------------------------------------------------------
    if (EPI == EPI_RESID) {
        float* xnew = (float*)(smem + 256) + (size_t)p.tpw * p.ks * NMAT * plane;   // [tpw][64][16]
        for (int it = tid; it < p.tpw * M * 16; it += blockDim.x) {
            const int t = it / (M * 16), rem = it - t * M * 16, m = rem >> 4, c = rem & 15;
            const int tg = blockIdx.x * p.tpw + t;
            if (tg >= p.tiles) continue;
            const int n = tg * 16 + c;
            float* x = p.X + (size_t)p.rows[m].xrow * p.g.h + n;
            const float v = *x + fin(t, 0, m, c);
            *x = v;
            xnew[(t * 64 + m) * 16 + c] = v;
            if (BF)
                ((uint16_t*)p.XBout)[(size_t)m * p.g.h + n] = f2bf(v);
            else
                ((float*)p.XBout)[(size_t)m * p.g.h + n] = v;
        }
        __syncthreads();
        for (int it = tid; it < p.tpw * M; it += blockDim.x) {
            const int t = it / M, m = it - t * M;
            const int tg = blockIdx.x * p.tpw + t;
            if (tg >= p.tiles) continue;
            p.SSQRout[(size_t)m * p.g.ssq_tiles + tg] = ssq16(&xnew[(t * 64 + m) * 16]);
        }
    } else if (EPI == EPI_SWIGLU) {
        for (int it = tid; it < p.tpw * M * 16; it += blockDim.x) {
            const int t = it / (M * 16), rem = it - t * M * 16, m = rem >> 4, c = rem & 15;
            const int tg = blockIdx.x * p.tpw + t;
            if (tg >= p.tiles) continue;
            const float gt = fin(t, 0, m, c), up = fin(t, NMAT - 1, m, c);
            const float a = gt / (1.0f + expf(-gt)) * up;
            const size_t o = (size_t)m * p.N_mat + tg * 16 + c;
            if (BF)
                ((uint16_t*)p.act)[o] = f2bf(a);
            else
                ((float*)p.act)[o] = a;
        }
    } else if (EPI == EPI_QKV) {
        const int tph = p.g.h / kTile, tpd = p.g.dh / kTile, half = p.g.dh / 2;
        for (int it = tid; it < p.tpw * M * 8; it += blockDim.x) {
            const int t = it / (M * 8), rem = it - t * M * 8, m = rem >> 3, c = rem & 7;
            const int tg = blockIdx.x * p.tpw + t;
            if (tg >= p.tiles) continue;
            const int mat = tg / tph, lt = tg - mat * tph, head = lt / tpd, sub = lt - head * tpd;
            const int i = sub * 8 + c;                      // pair (i, i + dh/2)
            const int pos = p.rows[m].pos;
            float x0 = fin(t, 0, m, c), x1 = fin(t, 0, m, c + 8);
            if (mat < 2) {
                const float cs = p.rope[((size_t)pos * half + i) * 2];
                const float sn = p.rope[((size_t)pos * half + i) * 2 + 1];
                const float y0 = x0 * cs - x1 * sn, y1 = x1 * cs + x0 * sn;
                x0 = y0;
                x1 = y1;
            }
            const int col = head * p.g.dh + i;
            if (mat == 0) {
                p.qout[(size_t)m * p.g.h + col] = x0;
                p.qout[(size_t)m * p.g.h + col + half] = x1;
            } else {
                const int slot = p.rows[m].slot;
                const int tb = kv_table(p.g, p.stack, p.layer, p.rows[m].depth);
                const int kv = mat - 1;
                WT* dst = (WT*)(slot >= 0 ? p.kvs : p.kvc) +
                          (slot >= 0 ? kvs_index(p.g, slot, tb, kv) : kvc_index(p.g, p.rows[m].seq, tb, kv, pos));
                if (BF) {
                    ((uint16_t*)dst)[col] = f2bf(x0);
                    ((uint16_t*)dst)[col + half] = f2bf(x1);
                } else {
                    ((float*)dst)[col] = x0;
                    ((float*)dst)[col + half] = x1;
                }
            }
        }
    } else if (EPI == EPI_LOGITS) {
        for (int it = tid; it < p.tpw * M * 16; it += blockDim.x) {
            const int t = it / (M * 16), rem = it - t * M * 16, m = rem >> 4, c = rem & 15;
            const int tg = blockIdx.x * p.tpw + t;
            const int n = tg * 16 + c;
            if (tg >= p.tiles || n >= p.N_mat) continue;
            const float v = fin(t, 0, m, c);
            p.logits[(size_t)m * p.N_mat + n] = v;
            if (!(fabsf(v) <= 3.0e38f)) atomicOr(p.err, 1);
        }
        for (int it = tid; it < p.tpw * M; it += blockDim.x) {
            const int t = it / M, m = it - t * M;
            const int tg = blockIdx.x * p.tpw + t;
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

// ---------------------------------------------------------------------------
// Weight packing (once, when the weights are bound): every wavefront load of
// the GEMM becomes one contiguous 1 KB block, with the RMSNorm gain folded in.
// ---------------------------------------------------------------------------
static int tiles_of(int epi, int N_mat) {
    const int t = (N_mat + kTile - 1) / kTile;
    return epi == EPI_QKV ? 3 * t : t;
}

size_t packed_elems(int epi, int N_mat, int K, bool) {
    const int nmat = epi == EPI_SWIGLU ? 2 : 1;
    return (size_t)tiles_of(epi, N_mat) * kTile * nmat * K;
}

template <typename WT, int EPI>
__global__ void __launch_bounds__(256) k_pack(const WT* W0, const WT* W1, const WT* W2, const WT* gain, WT* out,
                                              int N_mat, int K, Geo g, size_t n_vec) {
    constexpr int VEC = WTraits<WT>::VEC, KSTEP = WTraits<WT>::KSTEP;
    constexpr int NMAT = EPI == EPI_SWIGLU ? 2 : 1;
    const int nsteps = K / KSTEP;
    GemmParams p{};
    p.g = g;
    for (size_t v = (size_t)blockIdx.x * blockDim.x + threadIdx.x; v < n_vec; v += (size_t)gridDim.x * blockDim.x) {
        const int lane = (int)(v % 64);
        size_t r = v / 64;
        const int q = (int)(r % NMAT);
        r /= NMAT;
        const int s = (int)(r % nsteps);
        const int tile = (int)(r / nsteps);
        int mat = 0;
        const int row = tile_row<EPI>(p, tile, lane & 15, &mat);
        const WT* src = NMAT == 2 ? (q ? W1 : W0) : (mat == 0 ? W0 : mat == 1 ? W1 : W2);
        const int k0 = s * KSTEP + (lane >> 4) * VEC;
        WT* dst = out + v * VEC;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            float w = 0.f;
            if (row < N_mat) {
                w = sizeof(WT) == 2 ? bf2f(((const uint16_t*)src)[(size_t)row * K + k0 + e])
                                    : ((const float*)src)[(size_t)row * K + k0 + e];
                if (gain) w *= sizeof(WT) == 2 ? bf2f(((const uint16_t*)gain)[k0 + e]) : ((const float*)gain)[k0 + e];
            }
            if (sizeof(WT) == 2)
                ((uint16_t*)dst)[e] = f2bf(w);
            else
                ((float*)dst)[e] = w;
        }
    }
}

template <typename WT, int EPI>
static hipError_t pack_t(const void* const* W, const void* gain, void* out, int N_mat, int K, const Geo& g,
                         hipStream_t st) {
    constexpr int VEC = WTraits<WT>::VEC;
    const size_t n_vec = packed_elems(EPI, N_mat, K, sizeof(WT) == 2) / VEC;
    const int blocks = (int)std::min<size_t>((n_vec + 255) / 256, 65536);
    hipLaunchKernelGGL((k_pack<WT, EPI>), dim3(blocks), dim3(256), 0, st, (const WT*)W[0], (const WT*)W[1],
                       (const WT*)W[2], (const WT*)gain, (WT*)out, N_mat, K, g, n_vec);
    return hipGetLastError();
}

hipError_t launch_pack(int epi, const void* const* W, const void* gain, void* out, int N_mat, int K, const Geo& g,
                       bool bf16, hipStream_t st) {
    if (bf16) {
        switch (epi) {
            case EPI_QKV: return pack_t<uint16_t, EPI_QKV>(W, gain, out, N_mat, K, g, st);
            case EPI_RESID: return pack_t<uint16_t, EPI_RESID>(W, gain, out, N_mat, K, g, st);
            case EPI_SWIGLU: return pack_t<uint16_t, EPI_SWIGLU>(W, gain, out, N_mat, K, g, st);
            case EPI_LOGITS: return pack_t<uint16_t, EPI_LOGITS>(W, gain, out, N_mat, K, g, st);
        }
    } else {
        switch (epi) {
            case EPI_QKV: return pack_t<float, EPI_QKV>(W, gain, out, N_mat, K, g, st);
            case EPI_RESID: return pack_t<float, EPI_RESID>(W, gain, out, N_mat, K, g, st);
            case EPI_SWIGLU: return pack_t<float, EPI_SWIGLU>(W, gain, out, N_mat, K, g, st);
            case EPI_LOGITS: return pack_t<float, EPI_LOGITS>(W, gain, out, N_mat, K, g, st);
        }
    }
    return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------
size_t gemm_lds_bytes(int wbytes, int epi, int nmat, int tpw, int ks, int kc, int nt_max) {
    const int vec = wbytes == 2 ? 8 : 4;
    const size_t a = nt_max > 1 ? (size_t)nt_max * 16 * (kc + vec) * wbytes : 0;
    size_t r = (size_t)tpw * ks * nmat * nt_max * 256 * 4;
    if (epi == EPI_RESID) r += (size_t)tpw * 64 * 16 * 4;
    return 256 + (a > r ? a : r);
}

template <typename WT, int EPI, int NMAT, int NTM>
static hipError_t launch_t(const GemmParams& p, int nt_max, hipStream_t st) {
    const int nblk = (p.tiles + p.tpw - 1) / p.tpw;
    const size_t lds = gemm_lds_bytes(sizeof(WT), EPI, NMAT, p.tpw, p.ks, p.kc, nt_max);
    hipLaunchKernelGGL((k_gemm<WT, EPI, NMAT, NTM>), dim3(nblk), dim3(64 * p.tpw * p.ks), lds, st, p);
    return hipGetLastError();
}

template <typename WT, int EPI, int NMAT>
static hipError_t launch_n(const GemmParams& p, int nt_max, hipStream_t st) {
    return nt_max <= 1 ? launch_t<WT, EPI, NMAT, 1>(p, nt_max, st) : launch_t<WT, EPI, NMAT, 4>(p, nt_max, st);
}

template <typename WT, int EPI, int NMAT>
static hipError_t allow_lds(int bytes) {
    hipError_t a = hipFuncSetAttribute((const void*)k_gemm<WT, EPI, NMAT, 1>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    hipError_t b = hipFuncSetAttribute((const void*)k_gemm<WT, EPI, NMAT, 4>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    return a != hipSuccess ? a : b;
}

hipError_t gemm_prepare(int lds_bytes) {
    hipError_t e = hipSuccess;
    hipError_t r[] = {allow_lds<uint16_t, EPI_QKV, 1>(lds_bytes),  allow_lds<uint16_t, EPI_RESID, 1>(lds_bytes),
                      allow_lds<uint16_t, EPI_SWIGLU, 2>(lds_bytes), allow_lds<uint16_t, EPI_LOGITS, 1>(lds_bytes),
                      allow_lds<float, EPI_QKV, 1>(lds_bytes),     allow_lds<float, EPI_RESID, 1>(lds_bytes),
                      allow_lds<float, EPI_SWIGLU, 2>(lds_bytes),  allow_lds<float, EPI_LOGITS, 1>(lds_bytes)};
    for (hipError_t x : r)
        if (x != hipSuccess) e = x;
    return e;
}

hipError_t launch_gemm(const GemmParams& p, int epi, bool bf16, int nt_max, hipStream_t st) {
    if (bf16) {
        switch (epi) {
            case EPI_QKV: return launch_n<uint16_t, EPI_QKV, 1>(p, nt_max, st);
            case EPI_RESID: return launch_n<uint16_t, EPI_RESID, 1>(p, nt_max, st);
            case EPI_SWIGLU: return launch_n<uint16_t, EPI_SWIGLU, 2>(p, nt_max, st);
            case EPI_LOGITS: return launch_n<uint16_t, EPI_LOGITS, 1>(p, nt_max, st);
        }
    } else {
        switch (epi) {
            case EPI_QKV: return launch_n<float, EPI_QKV, 1>(p, nt_max, st);
            case EPI_RESID: return launch_n<float, EPI_RESID, 1>(p, nt_max, st);
            case EPI_SWIGLU: return launch_n<float, EPI_SWIGLU, 2>(p, nt_max, st);
            case EPI_LOGITS: return launch_n<float, EPI_LOGITS, 1>(p, nt_max, st);
        }
    }
    return hipErrorInvalidValue;
}

}  // namespace ls
