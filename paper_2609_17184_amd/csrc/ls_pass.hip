// Persistent pass kernel: every block of a stack over one row list in a single
// launch.
//
// With a handful of branch rows a decode step is a stream of small phases
// (per block: QKV, attention, O, gate/up, down) whose launch and drain costs
// rival their data movement.  Here one workgroup per CU stays resident for the
// whole pass; phases are separated by a device-wide barrier (below), and
// between arriving and waiting each workgroup already issues the weight loads
// of its next phase: weights do not depend on the activations, so the weight
// stream continues across phase boundaries.  Each phase uses the same work
// items and arithmetic as the standalone kernels.  A barrier that does not
// complete within its spin budget flags ERR_SYNC and lets every workgroup run
// to the end, so the launch always terminates.  The grid is one workgroup per
// CU, all co-resident (checked at set-up); the barrier counters are zero at
// launch (the gather kernel in front of every pass clears them).
#include "ls_pass.h"

#include <algorithm>

#include "ls_attn_dev.h"
#include "ls_gemm_dev.h"
#include "ls_sched.h"

#ifndef LS_PASS_ATTN_ITEMS
#define LS_PASS_ATTN_ITEMS 0
#endif

namespace ls {

// Device-wide barrier.  Every access to data that crosses workgroups inside
// the launch is device-scope (see ld_f32 / st_f32 and the COH paths of the
// GEMM and attention items), so no cache writeback or invalidation is needed:
// each wave waits for its own stores to complete, then one arrival per
// workgroup is counted on one of kBarSub counters (in separate cache lines, so
// arrivals do not serialise on one address), and wave 0 polls the sum.
__device__ __forceinline__ void pass_arrive(unsigned* ctr) {
    __builtin_amdgcn_s_waitcnt(0);                      // this wave's stores have completed
    __syncthreads();
    if (threadIdx.x == 0)
        __hip_atomic_fetch_add(ctr + (blockIdx.x % kBarSub) * kBarStride, 1u, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
}

// Wait until `target` arrivals are counted.  After a timeout (ERR_SYNC) no
// barrier of the launch waits any more, so the launch still ends.
__device__ __forceinline__ void pass_wait(unsigned* ctr, unsigned target, int32_t* err) {
    if (threadIdx.x < 64) {
        const int lane = threadIdx.x;
        if (!(__hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & ERR_SYNC)) {
            unsigned n = 0;
            for (;;) {
                unsigned v = lane < kBarSub
                                 ? __hip_atomic_load(ctr + lane * kBarStride, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                                 : 0u;
#pragma unroll
                for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
                if (v >= target) break;
                if (++n > (1u << 21)) {
                    if (lane == 0) atomicOr(err, ERR_SYNC);
                    break;
                }
            }
        }
    }
    __syncthreads();
}

template <typename WT, int DH>
__global__ void __launch_bounds__(kPassThreads) k_pass(PassParams pp) {
    extern __shared__ __align__(16) char smem[];
    const int M = *pp.qkv.nrows;
    if (M <= 0) return;
    const int G = gridDim.x, it = blockIdx.x, H = pp.attn.g.H;
    unsigned target = 0;
    constexpr int SQ = pass_max_steps(EPI_QKV), SR = pass_max_steps(EPI_RESID), SG = pass_max_steps(EPI_SWIGLU);
    // Work items of consecutive phases go to consecutive ranges of workgroups
    // (cyclically), so a workgroup idle in one phase is usually busy in the
    // next: it issues that phase's weight loads as soon as the current phase
    // starts.  idx(b) is this workgroup's item index in a phase whose first
    // item sits on workgroup b.
    auto idx = [&](int b) { return it >= b ? it - b : it - b + G; };
    // attention tasks (row, head, chunk of kChunk positions) of this pass
    int attn_tasks_n = 0;
    for (int m = 0; m < M; ++m) attn_tasks_n += H * (pp.attn.rows[m].pos / kChunk + 1);
#if LS_PASS_ATTN_ITEMS
    const int attn_slots = M * H < G ? M * H : G;
#else
    const int attn_slots = attn_tasks_n < G ? attn_tasks_n : G;
#endif
    int bq = 0;
    // Register sets are scoped to their phase and loaded unconditionally, so
    // only the set in flight is live (the QKV set carries over to the next block).
    BRegs<WT, 1, SQ> rq;
    GemmParams q = pp.qkv;
    q.Wp = pp.wl[0];
    q.layer = 0;
    gemm_load_b<WT, 1, SQ>(q, idx(bq), rq, idx(bq) < pp.items_qkv);
    for (int l = 0; l < pp.L; ++l) {
        const int ba = (bq + pp.items_qkv) % G;
        const int bo = (ba + attn_slots) % G;
        const int bg = (bo + pp.items_o) % G;
        const int bd = (bg + pp.items_gu) % G;
        const int bn = (bd + pp.items_down) % G;
        // ---- RMSNorm + QKV + RoPE + KV write (weights already in flight) -------
        q = pp.qkv;
        q.Wp = pp.wl[4 * l];
        q.layer = l;
        if (idx(bq) < pp.items_qkv) gemm_finish<WT, EPI_QKV, 1, SQ, true>(q, idx(bq), M, rq, smem);
        pass_arrive(pp.ctr);
        pass_wait(pp.ctr, target += G, pp.err);
        // ---- attention at every row's own depth ---------------------------------
        AttnParams a = pp.attn;
        a.layer = l;
#if LS_PASS_ATTN_ITEMS
        for (int x = idx(ba); x < M * H; x += G) attn_item<WT, DH, true>(a, x / H, x % H, (float*)smem);
#else
        attn_tasks<WT, DH>(a, M, idx(ba), G, pp.apart, pp.acnt);
#endif
        pass_arrive(pp.ctr);
        {   // ---- O projection + residual -----------------------------------------
            BRegs<WT, 1, SR> ro;
            GemmParams o = pp.o;
            o.Wp = pp.wl[4 * l + 1];
            const int x = idx(bo);
            gemm_load_b<WT, 1, SR>(o, x, ro, x < pp.items_o);
            pass_wait(pp.ctr, target += G, pp.err);
            if (x < pp.items_o) gemm_finish<WT, EPI_RESID, 1, SR, true>(o, x, M, ro, smem);
        }
        pass_arrive(pp.ctr);
        {   // ---- RMSNorm + gate/up + SwiGLU ---------------------------------------
            BRegs<WT, 2, SG> rg;
            GemmParams gu = pp.gu;
            gu.Wp = pp.wl[4 * l + 2];
            const int x = idx(bg);
            gemm_load_b<WT, 2, SG>(gu, x, rg, x < pp.items_gu);
            pass_wait(pp.ctr, target += G, pp.err);
            if (x < pp.items_gu) gemm_finish<WT, EPI_SWIGLU, 2, SG, true>(gu, x, M, rg, smem);
        }
        pass_arrive(pp.ctr);
        {   // ---- down projection + residual ---------------------------------------
            BRegs<WT, 1, SR> rd;
            GemmParams dn = pp.down;
            dn.Wp = pp.wl[4 * l + 3];
            const int x = idx(bd);
            gemm_load_b<WT, 1, SR>(dn, x, rd, x < pp.items_down);
            pass_wait(pp.ctr, target += G, pp.err);
            if (x < pp.items_down) gemm_finish<WT, EPI_RESID, 1, SR, true>(dn, x, M, rd, smem);
        }
        // ---- next block's QKV weights (none after the last block) -------------------
        const bool more = l + 1 < pp.L;
        bq = bn;
        if (more) pass_arrive(pp.ctr);
        GemmParams nq = pp.qkv;
        nq.Wp = pp.wl[more ? 4 * (l + 1) : 0];
        gemm_load_b<WT, 1, SQ>(nq, idx(bq), rq, more && idx(bq) < pp.items_qkv);
        if (more) pass_wait(pp.ctr, target += G, pp.err);
    }
}

size_t pass_lds_bytes(const PassParams& pp, int wbytes) {
    size_t m = 0;
    const GemmParams* g[4] = {&pp.qkv, &pp.o, &pp.gu, &pp.down};
    const int epi[4] = {EPI_QKV, EPI_RESID, EPI_SWIGLU, EPI_RESID};
    for (int k = 0; k < 4; ++k)
        m = std::max(m, gemm_lds_bytes(wbytes, epi[k], epi[k] == EPI_SWIGLU ? 2 : 1, g[k]->tpw, g[k]->ks, 32, 1));
    return std::max(m, attention_lds_bytes(pp.attn.chunks_cap, pp.attn.g.dh));
}

template <typename WT>
static const void* pass_fn(int dh) {
    switch (dh) {
        case 16: return (const void*)k_pass<WT, 16>;
        case 32: return (const void*)k_pass<WT, 32>;
        case 64: return (const void*)k_pass<WT, 64>;
    }
    if (sizeof(WT) == 2) {   // 16-byte head slices of at most 16 lanes
        if (dh == 96) return (const void*)k_pass<uint16_t, 96>;
        if (dh == 128) return (const void*)k_pass<uint16_t, 128>;
    }
    return nullptr;
}

hipError_t pass_prepare(int lds_bytes, bool bf16, int dh) {
    const void* f = bf16 ? pass_fn<uint16_t>(dh) : pass_fn<float>(dh);
    if (!f) return hipErrorInvalidValue;
    return hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
}

int pass_occupancy(bool bf16, int dh, int lds_bytes) {
    const void* f = bf16 ? pass_fn<uint16_t>(dh) : pass_fn<float>(dh);
    if (!f) return 0;
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, f, kPassThreads, lds_bytes) != hipSuccess) {
        (void)hipGetLastError();
        return 0;
    }
    return n;
}

template <typename WT>
static void launch_wt(const PassParams& pp, int grid, size_t lds, hipStream_t st) {
    switch (pp.attn.g.dh) {
        case 16: hipLaunchKernelGGL((k_pass<WT, 16>), dim3(grid), dim3(kPassThreads), lds, st, pp); break;
        case 32: hipLaunchKernelGGL((k_pass<WT, 32>), dim3(grid), dim3(kPassThreads), lds, st, pp); break;
        case 64: hipLaunchKernelGGL((k_pass<WT, 64>), dim3(grid), dim3(kPassThreads), lds, st, pp); break;
    }
}
static void launch_bf16(const PassParams& pp, int grid, size_t lds, hipStream_t st) {
    switch (pp.attn.g.dh) {
        case 96: hipLaunchKernelGGL((k_pass<uint16_t, 96>), dim3(grid), dim3(kPassThreads), lds, st, pp); break;
        case 128: hipLaunchKernelGGL((k_pass<uint16_t, 128>), dim3(grid), dim3(kPassThreads), lds, st, pp); break;
        default: launch_wt<uint16_t>(pp, grid, lds, st);
    }
}

hipError_t launch_pass(const PassParams& pp, bool bf16, int grid, hipStream_t st) {
    const size_t lds = pass_lds_bytes(pp, bf16 ? 2 : 4);
    if (bf16)
        launch_bf16(pp, grid, lds, st);
    else
        launch_wt<float>(pp, grid, lds, st);
    return hipGetLastError();
}

}  // namespace ls
