// Persistent pass kernel: one launch runs every block of a stack over a row
// list (ls_pass.hip).
#pragma once
#include "ls_attn.h"
#include "ls_gemm.h"

namespace ls {

constexpr int kPassThreads = 512;   // one 8-wave workgroup per CU: 256 VGPRs per lane
constexpr int kPassRows = 16;       // rows a persistent pass handles
// Attention inside the pass, chosen per handle from its context capacity:
// with at most kPassAttnWgChunks chunks per row, one workgroup per (row,
// head) whose waves combine their chunk partials in LDS; above it, (row, head,
// chunk) tasks over every wave of the chip, combined through device memory by
// the wave that completes a (row, head), so long contexts stream their keys
// and values on every CU.
constexpr int kPassAttnWgChunks = 32;

// Phases of a block in the pass.
enum PassKind { PK_QKV = 0, PK_O = 1, PK_GU = 2, PK_DOWN = 3 };
// k steps per wave a phase keeps in flight (register budget of 8 waves per CU).
// The O projection (K = h) gets 8 steps on models with h <= 2048 and 24
// ("wide" instantiation) above.
__host__ __device__ constexpr int pass_max_steps(int kind, bool wide) {
    return kind == PK_O ? (wide ? 24 : 16) : kind == PK_DOWN ? 24 : 16;
}

// Per-block activation buffers of one pass, each [kPassRows][width] row-major
// and written once per launch (filled with the sentinel before it):
//   XB[l], SSQ[l]   input of block l's QKV (rounded state, tile sums of squares);
//                   l = 0 comes from the row's X, l > 0 from block l-1's down
//   Q[l]            rotated queries                     (QKV -> attention)
//   ATT[l]          attention output                    (attention -> O)
//   XO[l]           residual after O, fp32              (O -> down)
//   XBO[l], SSQO[l] its rounded copy and sums of squares (O -> gate/up)
//   ACT[l]          SwiGLU activation                   (gate/up -> down)
//   XD[l]           residual after down, fp32          (down -> next O); the
//                   last block writes the rows' X instead
struct PassFlow {
    void* XB;       // [L+1][rows][h]    weight dtype
    float* SSQ;     // [L+1][rows][h/16]
    float* Q;       // [L][rows][h]
    void* ATT;      // [L][rows][h]      weight dtype
    float* XO;      // [L][rows][h]
    void* XBO;      // [L][rows][h]      weight dtype
    float* SSQO;    // [L][rows][h/16]
    void* ACT;      // [L][rows][F]      weight dtype
    float* XD;      // [L][rows][h]
};

// bytes of the flow buffers for `layers` blocks
size_t pass_flow_bytes(const Geo& g, int layers, int wbytes);
// carve a flow out of one allocation of pass_flow_bytes
PassFlow pass_flow_carve(void* base, const Geo& g, int layers, int wbytes);

struct PassParams {
    GemmParams qkv, o, gu, down;    // per-kind parameters; Wp, layer and buffers are set per block
    AttnParams attn;
    PassFlow flow;
    const void* const* wl;          // device: [L][4] packed weights (qkv, o, gate/up, down)
    int L;
    int stack;
    int attn_wg;                    // 1: attention per (row, head) workgroup; 0: chunk tasks (below)
    unsigned* acnt;                 // device: [kPassRows][H] attention counters (chunk tasks, or the parts of a
                                    // split (row, head) item), zero at launch
    float* apart;                   // device: [kPassRows][H][chunks_cap + 1][dh + 2] attention chunk partials
    int32_t* err;                   // kErrPoll when a read gave up waiting
    int items_qkv, items_o, items_gu, items_down;
    int lds_rows;                   // byte offset of the row table's copy in dynamic LDS (set by launch_pass)
    int lds_stage;                  // byte offset of the weight staging area in dynamic LDS, -1: none (set by launch_pass)
};

size_t pass_lds_bytes(const PassParams& pp, int wbytes);
// wide: the instantiation for h > 2048 (see pass_max_steps)
hipError_t pass_prepare(int lds_bytes, bool bf16, int dh, bool wide);
// Everything a launch needs before it starts: the flow buffers of the rows
// filled with the sentinel, XB[0] / SSQ[0] from the rows' X, the rows' own
// slot keys / values of every block of the stack filled with the sentinel,
// the attention counters zeroed.  rows_cap: the capacity of the row list.
hipError_t launch_pass_prep(const PassParams& pp, bool bf16, int rows_cap, hipStream_t st);
// grid = the number of co-resident workgroups (one per CU)
hipError_t launch_pass(const PassParams& pp, bool bf16, int grid, hipStream_t st);
// workgroups of k_pass one CU can hold (0 when it cannot be launched)
int pass_occupancy(bool bf16, int dh, bool wide, int lds_bytes);

}  // namespace ls
