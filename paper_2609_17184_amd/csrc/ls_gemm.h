// Launch interface of the weight-streaming skinny GEMM (ls_gemm.hip).
#pragma once
#include "ls_common.h"

namespace ls {

enum Epi { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_LOGITS = 3 };
enum AMode { A_NORM = 0, A_BUF = 1 };

// k steps (one 16-byte weight load per lane each) a wavefront keeps in flight
// for an epilogue kind and NTM 16-row tiles of accumulators (register budget:
// the residual GEMMs hold no RMSNorm statistics, gate/up streams two matrices)
__host__ __device__ constexpr int gemm_max_steps(int epi, int ntm) {
    return ntm > 1 ? (epi == EPI_SWIGLU ? 4 : 8) : (epi == EPI_RESID ? 12 : 8);
}

struct GemmParams {
    Geo g;
    const int32_t* nrows;      // device: number of rows M (<= 64)
    const Row* rows;           // device: row descriptors
    // activations (row order of the pass)
    // QKV, SWIGLU and LOGITS read A = XB and scale outputs by 1/rms from SSQR;
    // RESID reads A = abuf
    const void* XB;            // [M][K] compute dtype (fp16 for 16-bit models, else fp32)
    const float* SSQR;         // [M][h/16]
    const void* abuf;          // [M][K] compute dtype
    int K;
    // weights packed in MFMA operand order (see launch_pack): [tile][step][NMAT][64 lanes][16 bytes]
    const void* Wp;
    int N_mat;                 // output features per matrix
    int tiles;                 // 16-column tiles in the launch
    int tpw, ks, kc;           // tiles per workgroup, k-slices (waves) per workgroup, LDS k chunk (64-row variant)
    // split k across workgroups (direct path, tpw = 1): kg workgroups per tile,
    // each summing its ks slices; the last of them to finish (counted on
    // cnt[tile]) sums the kg partials in workgroup order and runs the
    // epilogue.  kg <= 1: one workgroup holds every slice of its tiles.
    int kg;
    float* part;               // [tiles * kg][NMAT][16 rows][16 cols] fp32 partials (kg > 1)
    unsigned* cnt;             // [tiles] arrival counters, zero between launches (kg > 1)
    // epilogue outputs
    float* X;                  // RESID: X[row.xrow] += result
    const float* Xin;          // RESID in the persistent pass: residual input [M][h] (NULL: X)
    float* Xout;               // RESID in the persistent pass: residual output [M][h] (NULL: X)
    void* XBout;               // RESID: rounded new state, row order (NULL: not needed)
    float* SSQRout;            // RESID: its per-tile sums of squares, row order
    void* act;                 // SWIGLU: [M][N_mat]
    float* qout;               // QKV: [M][h] rotated queries
    void* kvc;                 // QKV: committed KV cache
    void* kvs;                 // QKV: slot KV cache
    const float* rope;         // QKV: [max_ctx][dh/2][2] cos, sin
    int stack, layer;          // QKV: KV table of the block
    float* logits;             // LOGITS: [M][V]
    float* tmax;               // LOGITS: [M][tiles]
    int32_t* targ;             // LOGITS: [M][tiles]
    int32_t* err;              // LOGITS: bit 0 set on NaN/Inf; persistent pass: kErrPoll
};

// Pack up to 3 row-major matrices [N_mat][K] (the tiles of an epilogue kind) into
// MFMA operand order, multiplying column k by gain[k] (gain may be NULL):
// out[tile][step][q][lane][VEC] = W[row(tile, lane % 16)][step*KSTEP + (lane/16)*VEC + e] * gain.
// QKV tiles take matrices in order q, k, v with each tile holding RoPE pairs.
size_t packed_elems(int epi, int N_mat, int K, bool bf16);
// bf16 weights become fp16 copies; a value beyond the fp16 range sets bit 0 of *err (device)
hipError_t launch_pack(int epi, const void* const* W, const void* gain, void* out, int N_mat, int K, const Geo& g,
                       bool bf16, int32_t* err, hipStream_t st);

size_t gemm_lds_bytes(int wbytes, int epi, int nmat, int tpw, int ks, int kc, int nt_max, int kg = 1);
hipError_t gemm_prepare(int lds_bytes);   // allow the dynamic LDS size on every instantiation
hipError_t launch_gemm(const GemmParams& p, int epi, bool bf16, int nt_max, hipStream_t st);

// Stream-K launches of at most 16 rows (ls_gemm_sk.hip): the grid that keeps
// every workgroup resident, and the most waves a tile can be split over (the
// partial slots per tile: p.kg of a launch, p.part holds tiles x kg x NMAT x
// 256 floats, p.cnt one counter per tile).
hipError_t gemm_sk_shape(int epi, bool bf16, int nt, int tiles, int K, int* grid, int* contrib);
hipError_t launch_gemm_sk(const GemmParams& p, int epi, bool bf16, int nt, int grid, hipStream_t st);

}  // namespace ls
