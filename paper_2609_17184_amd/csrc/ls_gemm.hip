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
//     feeds v_mfma_f32_16x16x32_f16 from registers -- one memory round trip,
//     no LDS staging; k is split over several workgroups per tile when one
//     workgroup's waves cannot hold it; larger launches (prefill, 64 rows)
//     stage A through LDS;
//   * 16-bit models compute in fp16: weights arrive as bf16 and are packed
//     into fp16 copies; the activations and key/value caches are fp16;
//   * epilogues: QKV (RoPE on q and k, K/V written to the KV cache of the
//     row's own depth), RESID (residual add, rounded copy and per-16-column
//     sums of squares for the next RMSNorm), SWIGLU (silu(g) * u), LOGITS
//     (logits + per-tile max / arg-max for the vocabulary-sharded readout).
#include "ls_gemm_dev.h"

#include <algorithm>

namespace ls {

template <typename WT, int EPI, int NMAT, int NTM>
__global__ void __launch_bounds__(1024) k_gemm(GemmParams p) {
    extern __shared__ __align__(16) char smem[];
    const int M = ld_uniform(p.nrows);
    if (M <= 0) return;
    if constexpr (NTM == 1) {
        // ---- direct operands: every load of the wave issued at entry; k is
        //      split over kg workgroups per tile so that no wave holds more than
        //      MAXS steps (the launch configuration guarantees it) ----------------
        constexpr int MAXS = gemm_max_steps(EPI, 1);
        const int kg = gemm_kg(p), item = (int)blockIdx.x / kg, kgi = (int)blockIdx.x - item * kg;
        gemm_direct<WT, EPI, NMAT, MAXS>(p, item, kgi, M, smem);
    } else {
        // ---- activations staged through LDS (up to 64 rows), weights in rounds ---
        constexpr int KSTEP = WTraits<WT>::KSTEP, VEC = WTraits<WT>::VEC;
        constexpr int MAXS = gemm_max_steps(EPI, NTM);
        constexpr bool norm = EPI != EPI_RESID;
        constexpr int NSS = norm ? 4 : 1;
        const WaveGeo w = wave_geo<WT, false>(p, blockIdx.x);
        const int tid = threadIdx.x, nt = (M + 15) >> 4;
        float ssv[NSS];
#pragma unroll
        for (int u = 0; u < NSS; ++u) {
            const int t = w.lane + 64 * u;
            ssv[u] = (norm && w.wave < M && t < p.g.ssq_tiles) ? p.SSQR[(size_t)w.wave * p.g.ssq_tiles + t] : 0.f;
        }
        const WT* Abase = (const WT*)(norm ? p.XB : p.abuf);
        const WT* bt = packed_tile<WT, NMAT>(p, w);
        f32x4 acc[NTM][NMAT];
#pragma unroll
        for (int rt = 0; rt < NTM; ++rt)
#pragma unroll
            for (int q = 0; q < NMAT; ++q) acc[rt][q] = f32x4{0.f, 0.f, 0.f, 0.f};
        WT* A = (WT*)(smem + 256);                           // [nt*16][astride]
        const int astride = p.kc + VEC;                      // 16-byte row pad
        const int span = MAXS * p.ks;
        for (int r0 = 0; r0 < w.nsteps; r0 += span) {
            const int ibase = r0 / p.ks;
            u32x4 b[MAXS][NMAT];
#pragma unroll
            for (int i = 0; i < MAXS; ++i) {
                const int s = w.ksl + (ibase + i) * p.ks;
#pragma unroll
                for (int q = 0; q < NMAT; ++q)
                    b[i][q] = (ibase + i < w.nst && w.tile_ok)
                                  ? __builtin_nontemporal_load((const u32x4*)(bt + ((size_t)s * NMAT + q) * 64 * VEC))
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
                if (!w.tile_ok) continue;
                const int s_lo = c0 / KSTEP, s_hi = (c0 + kc) / KSTEP;
#pragma unroll
                for (int i = 0; i < MAXS; ++i) {
                    const int ss = w.ksl + (ibase + i) * p.ks;
                    if (ibase + i >= w.nst || ss < s_lo || ss >= s_hi) continue;
                    const int ko = (ss - s_lo) * KSTEP + w.grp * VEC;
#pragma unroll
                    for (int rt = 0; rt < NTM; ++rt) {
                        if (rt >= nt) break;
                        const u32x4 a = *(const u32x4*)(A + (rt * 16 + w.j) * astride + ko);
                        mfma_step<WT, NMAT>(a, b[i], acc[rt]);
                    }
                }
            }
        }
        gemm_epilogue<WT, EPI, NMAT, NTM, NSS>(p, blockIdx.x, M, w, acc, ssv, smem);
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

// bf16 models: the copy is fp16 (the kernels' 16-bit compute type); a value
// outside the fp16 range sets bit 0 of *err.
template <typename WT, int EPI>
__global__ void __launch_bounds__(256) k_pack(const WT* W0, const WT* W1, const WT* W2, const WT* gain, WT* out,
                                              int N_mat, int K, Geo g, size_t n_vec, int32_t* err) {
    constexpr int VEC = WTraits<WT>::VEC, KSTEP = WTraits<WT>::KSTEP;
    constexpr int NMAT = EPI == EPI_SWIGLU ? 2 : 1;
    const int nsteps = K / KSTEP;
    for (size_t v = (size_t)blockIdx.x * blockDim.x + threadIdx.x; v < n_vec; v += (size_t)gridDim.x * blockDim.x) {
        const int lane = (int)(v % 64);
        size_t r = v / 64;
        const int q = (int)(r % NMAT);
        r /= NMAT;
        const int s = (int)(r % nsteps);
        const int tile = (int)(r / nsteps);
        int mat = 0;
        const int row = tile_row<EPI>(g, tile, lane & 15, &mat);
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
            if (sizeof(WT) == 2) {
                if (!(fabsf(w) <= kF16Max)) atomicOr(err, 1);
                ((uint16_t*)dst)[e] = f2h(w);
            } else {
                ((float*)dst)[e] = w;
            }
        }
    }
}

template <typename WT, int EPI>
static hipError_t pack_t(const void* const* W, const void* gain, void* out, int N_mat, int K, const Geo& g,
                         int32_t* err, hipStream_t st) {
    constexpr int VEC = WTraits<WT>::VEC;
    const size_t n_vec = packed_elems(EPI, N_mat, K, sizeof(WT) == 2) / VEC;
    const int blocks = (int)std::min<size_t>((n_vec + 255) / 256, 65536);
    hipLaunchKernelGGL((k_pack<WT, EPI>), dim3(blocks), dim3(256), 0, st, (const WT*)W[0], (const WT*)W[1],
                       (const WT*)W[2], (const WT*)gain, (WT*)out, N_mat, K, g, n_vec, err);
    return hipGetLastError();
}

hipError_t launch_pack(int epi, const void* const* W, const void* gain, void* out, int N_mat, int K, const Geo& g,
                       bool bf16, int32_t* err, hipStream_t st) {
    if (bf16) {
        switch (epi) {
            case EPI_QKV: return pack_t<uint16_t, EPI_QKV>(W, gain, out, N_mat, K, g, err, st);
            case EPI_RESID: return pack_t<uint16_t, EPI_RESID>(W, gain, out, N_mat, K, g, err, st);
            case EPI_SWIGLU: return pack_t<uint16_t, EPI_SWIGLU>(W, gain, out, N_mat, K, g, err, st);
            case EPI_LOGITS: return pack_t<uint16_t, EPI_LOGITS>(W, gain, out, N_mat, K, g, err, st);
        }
    } else {
        switch (epi) {
            case EPI_QKV: return pack_t<float, EPI_QKV>(W, gain, out, N_mat, K, g, err, st);
            case EPI_RESID: return pack_t<float, EPI_RESID>(W, gain, out, N_mat, K, g, err, st);
            case EPI_SWIGLU: return pack_t<float, EPI_SWIGLU>(W, gain, out, N_mat, K, g, err, st);
            case EPI_LOGITS: return pack_t<float, EPI_LOGITS>(W, gain, out, N_mat, K, g, err, st);
        }
    }
    return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------
size_t gemm_lds_bytes(int wbytes, int epi, int nmat, int tpw, int ks, int kc, int nt_max, int kg) {
    const int vec = wbytes == 2 ? 8 : 4;
    const size_t a = nt_max > 1 ? (size_t)nt_max * 16 * (kc + vec) * wbytes : 0;
    const int slices = std::max(tpw * ks, kg);          // the split-k finish holds kg partials
    size_t r = (size_t)slices * nmat * nt_max * 256 * 4;
    return 256 + (a > r ? a : r);
}

template <typename WT, int EPI, int NMAT, int NTM>
static hipError_t launch_t(const GemmParams& p, int nt_max, hipStream_t st) {
    const int kg = gemm_kg(p);
    if (kg > 1 && (NTM != 1 || p.tpw != 1 || kg > 16 || !p.part || !p.cnt)) return hipErrorInvalidValue;
    const int nblk = (p.tiles + p.tpw - 1) / p.tpw * kg;
    const size_t lds = gemm_lds_bytes(sizeof(WT), EPI, NMAT, p.tpw, p.ks, p.kc, nt_max, kg);
    GemmParams q = p;
    void* args[] = {(void*)&q};
    return ls_launch((const void*)k_gemm<WT, EPI, NMAT, NTM>, dim3(nblk), dim3(64 * p.tpw * p.ks), args, lds, st);
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
