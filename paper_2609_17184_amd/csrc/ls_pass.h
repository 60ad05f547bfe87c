// Persistent pass kernel: one launch runs every block of a stack over a row
// list (ls_pass.hip).
#pragma once
#include "ls_attn.h"
#include "ls_gemm.h"

namespace ls {

constexpr int kPassThreads = 512;   // one 8-wave workgroup per CU: 256 VGPRs per lane

// k steps per wave a pass phase keeps in flight (register budget of 8 waves per CU)
__host__ __device__ constexpr int pass_max_steps(int epi) { return epi == EPI_RESID ? 24 : 16; }

struct PassParams {
    GemmParams qkv, o, gu, down;    // per-kind parameters; Wp and layer are set per block
    AttnParams attn;
    const void* const* wl;          // device: [L][4] packed weights (qkv, o, gate/up, down)
    int L;
    unsigned* ctr;                  // device: barrier counters (kBarSub lines), zero at launch
    unsigned* acnt;                 // device: [16][H] attention chunk counters, zero at launch
    float* apart;                   // device: [16][H][chunks_cap][dh + 2] attention chunk partials
    int32_t* err;                   // ERR_SYNC on a barrier that timed out
    int items_qkv, items_o, items_gu, items_down;
};

size_t pass_lds_bytes(const PassParams& pp, int wbytes);
hipError_t pass_prepare(int lds_bytes, bool bf16, int dh);
// grid = the number of co-resident workgroups (one per CU)
hipError_t launch_pass(const PassParams& pp, bool bf16, int grid, hipStream_t st);
// workgroups of k_pass one CU can hold (0 when it cannot be launched)
int pass_occupancy(bool bf16, int dh, int lds_bytes);

}  // namespace ls
