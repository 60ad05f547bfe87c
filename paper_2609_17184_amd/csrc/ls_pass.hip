// Persistent pass kernel: every block of a stack over one row list in a single
// launch, synchronised by the data itself.
//
// With a handful of branch rows a decode step is a chain of small phases
// (per block: QKV, attention, O, gate/up, down) whose launch, drain and
// synchronisation costs rival their data movement.  Here one workgroup per CU
// stays resident for the whole pass and there is no barrier between phases:
// every activation a phase produces goes to a per-block buffer that was filled
// with a sentinel before the launch and is written once (ls_common.h), and a
// consumer reads its operands with device-scope loads until none is the
// sentinel.  A phase therefore starts on a workgroup as soon as the operands
// it needs exist, the producer never waits for its own stores, and the weight
// loads of a workgroup's next phase (which depend on nothing) are issued as
// soon as it finishes the current one.  Work items of consecutive phases go
// to consecutive ranges of workgroups, so a workgroup idle in one phase
// streams the next phase's weights early.  Each phase uses the same work items
// and arithmetic as the standalone kernels; reads that do not see their data
// within the spin budget set kErrPoll and stop waiting, so the launch always
// ends.  The grid is one workgroup per CU, all co-resident (checked at set-up);
// a workgroup only ever waits for data of earlier phases, which every other
// workgroup produces without waiting on it.
#include "ls_pass.h"

#include <algorithm>

#include "ls_attn_dev.h"
#include "ls_gemm_dev.h"
#include "ls_sched.h"

namespace ls {

static size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

size_t pass_flow_bytes(const Geo& g, int layers, int wbytes) {
    const size_t R = kPassRows, h = g.h, F = g.F, st = h / 16;
    size_t b = 0;
    b += align256((layers + 1) * R * h * wbytes);       // XB
    b += align256((layers + 1) * R * st * 4);           // SSQ
    b += align256(layers * R * h * 4);                  // Q
    b += align256(layers * R * h * wbytes);             // ATT
    b += align256(layers * R * h * 4);                  // XO
    b += align256(layers * R * h * wbytes);             // XBO
    b += align256(layers * R * st * 4);                 // SSQO
    b += align256(layers * R * F * wbytes);             // ACT
    b += align256(layers * R * h * 4);                  // XD
    return b;
}

PassFlow pass_flow_carve(void* base, const Geo& g, int layers, int wbytes) {
    const size_t R = kPassRows, h = g.h, F = g.F, st = h / 16;
    char* c = (char*)base;
    PassFlow f;
    auto take = [&](size_t bytes) {
        char* p = c;
        c += align256(bytes);
        return (void*)p;
    };
    f.XB = take((layers + 1) * R * h * wbytes);
    f.SSQ = (float*)take((layers + 1) * R * st * 4);
    f.Q = (float*)take(layers * R * h * 4);
    f.ATT = take(layers * R * h * wbytes);
    f.XO = (float*)take(layers * R * h * 4);
    f.XBO = take(layers * R * h * wbytes);
    f.SSQO = (float*)take(layers * R * st * 4);
    f.ACT = take(layers * R * F * wbytes);
    f.XD = (float*)take(layers * R * h * 4);
    return f;
}

// ---------------------------------------------------------------------------
// preparation of a launch (grid: rows_cap x kPrepY workgroups)
// ---------------------------------------------------------------------------
constexpr int kPrepY = 128;

template <typename WT>
__global__ void __launch_bounds__(256) k_pass_prep(PassParams pp) {
    const Geo& g = pp.qkv.g;
    const int m = blockIdx.x;
    if (m == 0 && blockIdx.y == 0)
        for (int i = threadIdx.x; i < kPassRows * g.H; i += blockDim.x) pp.acnt[i] = 0u;
    if (m >= *pp.qkv.nrows) return;
    const Row* rows = pp.qkv.rows;
    const size_t R = kPassRows, h = g.h, F = g.F, st = g.ssq_tiles;
    const PassFlow& f = pp.flow;
    if (blockIdx.y == 0) {
        // block 0's input: the row's state rounded, and its tile sums of squares
        const float* x = pp.qkv.X + (size_t)rows[m].xrow * h;
        for (int t = threadIdx.x; t < (int)st; t += blockDim.x) {
            float v[16];
#pragma unroll
            for (int c = 0; c < 16; ++c) v[c] = x[t * 16 + c];
            f.SSQ[(size_t)m * st + t] = f_value(ssq16(v));
#pragma unroll
            for (int c = 0; c < 16; ++c) {
                if (sizeof(WT) == 2)
                    ((uint16_t*)f.XB)[(size_t)m * h + t * 16 + c] = h_value(v[c]);
                else
                    ((float*)f.XB)[(size_t)m * h + t * 16 + c] = f_value(v[c]);
            }
        }
    }
    // sentinel over the row's slice of every per-block buffer, and over the
    // row's own slot keys / values of every block (written by this launch)
    const int slot = rows[m].slot, depth = rows[m].depth;
    constexpr int KINDS = 11;
    for (int seg = blockIdx.y; seg < KINDS * pp.L; seg += gridDim.y) {
        const int l = seg / KINDS, kind = seg - l * KINDS;
        uint32_t* p = nullptr;
        size_t words = 0;
        const size_t wb = sizeof(WT);
        switch (kind) {
            case 0: p = (uint32_t*)((char*)f.XB + ((l + 1) * R + m) * h * wb); words = h * wb / 4; break;
            case 1: p = (uint32_t*)(f.SSQ + ((l + 1) * R + m) * st); words = st; break;
            case 2: p = (uint32_t*)(f.Q + (l * R + m) * h); words = h; break;
            case 3: p = (uint32_t*)((char*)f.ATT + (l * R + m) * h * wb); words = h * wb / 4; break;
            case 4: p = (uint32_t*)(f.XO + (l * R + m) * h); words = h; break;
            case 5: p = (uint32_t*)((char*)f.XBO + (l * R + m) * h * wb); words = h * wb / 4; break;
            case 6: p = (uint32_t*)(f.SSQO + (l * R + m) * st); words = st; break;
            case 7: p = (uint32_t*)((char*)f.ACT + (l * R + m) * F * wb); words = F * wb / 4; break;
            case 8: p = (uint32_t*)(f.XD + (l * R + m) * h); words = h; break;
            default:
                if (slot >= 0) {
                    const int t = kv_table(g, pp.stack, l, depth);
                    p = (uint32_t*)((WT*)pp.qkv.kvs + kvs_index(g, slot, t, kind - 9));
                    words = h * wb / 4;
                }
        }
        for (size_t i = threadIdx.x; i < words; i += blockDim.x) p[i] = kSentinel;
    }
}

hipError_t launch_pass_prep(const PassParams& pp, bool bf16, int rows_cap, hipStream_t st) {
    if (bf16)
        hipLaunchKernelGGL(k_pass_prep<uint16_t>, dim3(rows_cap, kPrepY), dim3(256), 0, st, pp);
    else
        hipLaunchKernelGGL(k_pass_prep<float>, dim3(rows_cap, kPrepY), dim3(256), 0, st, pp);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// the pass
// ---------------------------------------------------------------------------
template <typename WT, int DH, bool WIDE>
__global__ void __launch_bounds__(kPassThreads) k_pass(PassParams pp) {
    extern __shared__ __align__(16) char smem[];
    const int M = *pp.qkv.nrows;
    if (M <= 0) return;
    if (M > kPassRows) {            // the launch never allows it; refuse rather than overrun LDS
        if (threadIdx.x == 0) atomicOr(pp.err, kErrPoll);
        return;
    }
    // The row table does not change during the pass.  A copy in LDS keeps its
    // reads (row positions, slots, depths, ancestors in every epilogue and
    // attention task) off the vector memory counter, which would order them
    // behind every weight load and store still outstanding.
    Row* lrows = (Row*)(smem + pp.lds_rows);
    for (int i = threadIdx.x; i < M * (int)(sizeof(Row) / 4); i += blockDim.x)
        ((uint32_t*)lrows)[i] = ((const uint32_t*)pp.qkv.rows)[i];
    __syncthreads();
    const int G = gridDim.x, it = blockIdx.x, H = pp.attn.g.H;
    const size_t R = kPassRows, h = pp.attn.g.h, F = pp.attn.g.F, st = pp.attn.g.ssq_tiles;
    const PassFlow& f = pp.flow;
    constexpr int SQ = pass_max_steps(PK_QKV, WIDE), SO = pass_max_steps(PK_O, WIDE);
    constexpr int SG = pass_max_steps(PK_GU, WIDE), SD = pass_max_steps(PK_DOWN, WIDE);
    // idx(b): this workgroup's item index in a phase whose first item sits on
    // workgroup b (phases take consecutive ranges of workgroups, cyclically)
    auto idx = [&](int b) { return it >= b ? it - b : it - b + G; };
    // attention items: (row, head, part) -- a row with more partials than the
    // workgroup has waves is split into parts of one partial per wave, unless
    // only its own position's partial is left over (a one-position second
    // round costs less than the hand-over) -- or (row, head, chunk) tasks
    const int AW = kPassThreads / 64;
    auto attn_parts = [&](int m) {
        const int n = (lrows[m].pos + kChunk - 1) / kChunk + 1;
        return n <= AW + 1 ? 1 : (n + AW - 1) / AW;
    };
    int attn_items = 0;
    for (int m = 0; m < M; ++m) attn_items += H * attn_parts(m);
    if (!pp.attn_wg) {
        attn_items = 0;
        for (int m = 0; m < M; ++m) attn_items += H * (lrows[m].pos / kChunk + 1);
    }
    const int attn_slots = attn_items < G ? attn_items : G;
    int bq = 0;
    // Weight staging: a workgroup with items in both gate/up and down would
    // otherwise start the down item's weight stream only once the gate/up item
    // is done.  Instead its waves stage the down item's first fragments in LDS
    // right after issuing the gate/up weights, before polling their operands,
    // and load them from LDS when the down phase comes.  The gate/up operand
    // wait covers the staging loads (loads complete in issue order).  Staging
    // the next block's QKV weights during the down phase, or the gate/up
    // weights during the O projection, measured slower: it delays the operand
    // reads of a phase on the critical path and adds to the bytes one CU
    // ingests there, while those weights have the time of a later wait anyway.
    const bool stage = pp.lds_stage >= 0;
    char* lds_wave = smem + (stage ? pp.lds_stage : 0) + (threadIdx.x >> 6) * (kPfFrags * 1024);
    bool staged_d = false;   // the down item's first fragments sit in LDS
    // Register sets are scoped to their phase and loaded unconditionally, so
    // only the set in flight is live (the QKV set carries over to the next block).
    BRegs<WT, 1, SQ> rq;
    GemmParams q = pp.qkv;
    q.rows = lrows;
    q.Wp = ld_uniform(pp.wl);
    gemm_load_b<WT, 1, SQ>(q, idx(bq), rq, idx(bq) < pp.items_qkv);
    for (int l = 0; l < pp.L; ++l) {
        const int ba = (bq + pp.items_qkv) % G;
        const int bo = (ba + attn_slots) % G;
        const int bg = (bo + pp.items_o) % G;
        const int bd = (bg + pp.items_gu) % G;
        const int bn = (bd + pp.items_down) % G;
        const bool last = l + 1 == pp.L;
        WT* XB = (WT*)f.XB + l * R * h;
        float* SSQ = f.SSQ + l * R * st;
        float* Q = f.Q + l * R * h;
        WT* ATT = (WT*)f.ATT + l * R * h;
        float* XO = f.XO + l * R * h;
        WT* XBO = (WT*)f.XBO + l * R * h;
        float* SSQO = f.SSQO + l * R * st;
        WT* ACT = (WT*)f.ACT + l * R * F;
        float* XD = f.XD + l * R * h;
        // ---- RMSNorm + QKV + RoPE + KV write (weights already in flight) -------
        q = pp.qkv;
        q.rows = lrows;
        q.Wp = ld_uniform(pp.wl + 4 * l);
        q.layer = l;
        q.XB = XB;
        q.SSQR = SSQ;
        q.qout = Q;
        if (idx(bq) < pp.items_qkv) gemm_finish<WT, EPI_QKV, 1, SQ, true>(q, idx(bq), M, rq, smem);
        __builtin_amdgcn_sched_barrier(0);
        // ---- attention at every row's own depth ---------------------------------
        AttnParams a = pp.attn;
        a.rows = lrows;
        a.layer = l;
        a.q = Q;
        a.out = ATT;
        if (pp.attn_wg) {
            for (int x = idx(ba); x < attn_items; x += G) {
                int m = 0, r = x;
                for (; m + 1 < M && r >= H * attn_parts(m); ++m) r -= H * attn_parts(m);
                const int parts = attn_parts(m), head = r / parts, part = r - head * parts;
                if (parts == 1)
                    attn_item<WT, DH, true>(a, m, head, (float*)smem);
                else
                    attn_item_part<WT, DH>(a, m, head, part, parts, pp.apart, pp.acnt, (float*)smem);
            }
        } else {
            attn_tasks<WT, DH>(a, M, idx(ba), G, pp.apart, pp.acnt);
        }
        __builtin_amdgcn_sched_barrier(0);
        {   // ---- O projection + residual -----------------------------------------
            BRegs<WT, 1, SO> ro;
            GemmParams o = pp.o;
            o.rows = lrows;
            o.Wp = ld_uniform(pp.wl + 4 * l + 1);
            o.abuf = ATT;
            o.Xin = l ? f.XD + (l - 1) * R * h : nullptr;
            o.Xout = XO;
            o.XBout = XBO;
            o.SSQRout = SSQO;
            const int x = idx(bo);
            gemm_load_b<WT, 1, SO>(o, x, ro, x < pp.items_o);
            __builtin_amdgcn_sched_barrier(0);
            if (x < pp.items_o) gemm_finish<WT, EPI_RESID, 1, SO, true>(o, x, M, ro, smem);
        }
        __builtin_amdgcn_sched_barrier(0);
        {   // ---- RMSNorm + gate/up + SwiGLU ---------------------------------------
            BRegs<WT, 2, SG> rg;
            GemmParams gu = pp.gu;
            gu.rows = lrows;
            gu.Wp = ld_uniform(pp.wl + 4 * l + 2);
            gu.XB = XBO;
            gu.SSQR = SSQO;
            gu.act = ACT;
            const int x = idx(bg), xd = idx(bd);
            gemm_load_b<WT, 2, SG>(gu, x, rg, x < pp.items_gu);
            staged_d = stage && x < pp.items_gu && xd < pp.items_down;
            if (staged_d) {
                GemmParams n = pp.down;
                n.Wp = ld_uniform(pp.wl + 4 * l + 3);
                __builtin_amdgcn_sched_barrier(0);
                gemm_stage_b<WT, 1, SD>(n, xd, lds_wave);
            }
            __builtin_amdgcn_sched_barrier(0);
            if (x < pp.items_gu) gemm_finish<WT, EPI_SWIGLU, 2, SG, true>(gu, x, M, rg, smem);
        }
        __builtin_amdgcn_sched_barrier(0);
        {   // ---- down projection + residual ---------------------------------------
            BRegs<WT, 1, SD> rd;
            GemmParams dn = pp.down;
            dn.rows = lrows;
            dn.Wp = ld_uniform(pp.wl + 4 * l + 3);
            dn.abuf = ACT;
            dn.Xin = XO;
            dn.Xout = last ? nullptr : XD;                 // the last block writes the rows' X
            dn.XBout = last ? nullptr : XB + R * h;
            dn.SSQRout = last ? nullptr : SSQ + R * st;
            const int x = idx(bd);
            if (staged_d)
                gemm_load_b_staged<WT, 1, SD>(dn, x, rd, lds_wave);
            else
                gemm_load_b<WT, 1, SD>(dn, x, rd, x < pp.items_down);
            __builtin_amdgcn_sched_barrier(0);
            if (x < pp.items_down) gemm_finish<WT, EPI_RESID, 1, SD, true>(dn, x, M, rd, smem);
        }
        __builtin_amdgcn_sched_barrier(0);
        // ---- next block's QKV weights (none after the last block) -------------------
        bq = bn;
        GemmParams nq = pp.qkv;
        nq.rows = lrows;
        nq.Wp = ld_uniform(pp.wl + (last ? 0 : 4 * (l + 1)));
        gemm_load_b<WT, 1, SQ>(nq, idx(bq), rq, !last && idx(bq) < pp.items_qkv);
    }
}

// LDS of the GEMM epilogues; the row table's copy follows it
static size_t pass_lds_gemm(const PassParams& pp, int wbytes) {
    size_t m = 0;
    const GemmParams* g[4] = {&pp.qkv, &pp.o, &pp.gu, &pp.down};
    const int epi[4] = {EPI_QKV, EPI_RESID, EPI_SWIGLU, EPI_RESID};
    for (int k = 0; k < 4; ++k)
        m = std::max(m, gemm_lds_bytes(wbytes, epi[k], epi[k] == EPI_SWIGLU ? 2 : 1, g[k]->tpw, g[k]->ks, 32, 1));
    if (pp.attn_wg) m = std::max(m, attention_lds_bytes(pp.attn.chunks_cap, pp.attn.g.dh));
    return (m + 15) & ~(size_t)15;
}

// weight staging: kPfFrags fragments of 1 KB per wave, when it fits in LDS
constexpr size_t kStageBytes = (size_t)(kPassThreads / 64) * kPfFrags * 1024;
static size_t pass_lds_base(const PassParams& pp, int wbytes) {
    return pass_lds_gemm(pp, wbytes) + kPassRows * sizeof(Row);
}
static bool pass_stage_fits(const PassParams& pp, int wbytes) {
    return pass_lds_base(pp, wbytes) + kStageBytes <= 160 * 1024;
}
size_t pass_lds_bytes(const PassParams& pp, int wbytes) {
    return pass_lds_base(pp, wbytes) + (pass_stage_fits(pp, wbytes) ? kStageBytes : 0);
}

template <typename WT, bool WIDE>
static const void* pass_fn_w(int dh) {
    switch (dh) {
        case 16: return (const void*)k_pass<WT, 16, WIDE>;
        case 32: return (const void*)k_pass<WT, 32, WIDE>;
        case 64: return (const void*)k_pass<WT, 64, WIDE>;
    }
    if constexpr (sizeof(WT) == 2) {   // 16-byte head slices of at most 16 lanes
        if (dh == 96) return (const void*)k_pass<WT, 96, WIDE>;
        if (dh == 128) return (const void*)k_pass<WT, 128, WIDE>;
    }
    return nullptr;
}

static const void* pass_fn(bool bf16, int dh, bool wide) {
    if (bf16) return wide ? pass_fn_w<uint16_t, true>(dh) : pass_fn_w<uint16_t, false>(dh);
    return wide ? pass_fn_w<float, true>(dh) : pass_fn_w<float, false>(dh);
}

hipError_t pass_prepare(int lds_bytes, bool bf16, int dh, bool wide) {
    const void* f = pass_fn(bf16, dh, wide);
    if (!f) return hipErrorInvalidValue;
    return hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
}

int pass_occupancy(bool bf16, int dh, bool wide, int lds_bytes) {
    const void* f = pass_fn(bf16, dh, wide);
    if (!f) return 0;
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, f, kPassThreads, lds_bytes) != hipSuccess) {
        (void)hipGetLastError();
        return 0;
    }
    return n;
}

hipError_t launch_pass(const PassParams& pp, bool bf16, int grid, hipStream_t st) {
    const size_t lds = pass_lds_bytes(pp, bf16 ? 2 : 4);
    const void* f = pass_fn(bf16, pp.attn.g.dh, pp.attn.g.h > 2048);
    if (!f) return hipErrorInvalidValue;
    PassParams q = pp;
    q.lds_rows = (int)pass_lds_gemm(pp, bf16 ? 2 : 4);
    q.lds_stage = pass_stage_fits(pp, bf16 ? 2 : 4) ? (int)pass_lds_base(pp, bf16 ? 2 : 4) : -1;
    void* args[] = {(void*)&q};
    return ls_launch(f, dim3(grid), dim3(kPassThreads), args, lds, st);
}

}  // namespace ls
