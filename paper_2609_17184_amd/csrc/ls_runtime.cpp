// Host runtime of the LoopSpec library: the C ABI of include/loopspec.h.
//
// A handle owns every device buffer (allocated once at create time), the
// launch configuration of each kernel, and the hipGraph of one decode step.
// One step = one batched pass of the shared blocks over every live branch
// (Sec. 4.2, Batched Recurrence), the readouts of the branches that reached a
// readout depth, the scheduler (Spawn / Verify / Reroot of Alg. 1), the KV
// commit of verified roots and the embedding (+ prelude) of spawned branches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/loopspec.h"
#include "ls_attn.h"
#include "ls_gemm.h"
#include "ls_pass.h"
#include "ls_sample.h"
#include "ls_sched.h"

namespace ls {
hipError_t launch_finalize_greedy(const Sched& s, int fin_op, const float* tmax, const int32_t* targ, int tiles,
                                  int rows_cap, hipStream_t st);
}  // namespace ls

using namespace ls;

namespace {

constexpr int kPrefillRows = 64;
constexpr size_t kLdsBudget = 80 * 1024;     // preferred GEMM workgroup LDS (two workgroups per CU)
constexpr size_t kLdsMax = 160 * 1024;       // LDS of one CU: the hard limit of a workgroup
constexpr size_t kSkWideBytes = 64u << 20;   // weight bytes from which launches of 17..64 rows run stream-K

struct GemmCfg {
    int ks = 1, tpw = 1, kc = 32, kg = 1;
    bool ok = true;
    // stream-K launches of 16, 32 and 64 rows (index 0, 1, 2): grid and
    // partial slots per tile (grid 0: that width takes the tiled GEMM)
    int sk_grid[3] = {0, 0, 0}, sk_c[3] = {0, 0, 0};
};

// Direct-path launch shape targets: about 16 waves per CU over the chip, and
// at least two workgroups per CU when the output tiles alone give fewer.
constexpr int kWaveTarget = 256 * 16;
constexpr int kWgTarget = 512;

// Worst-case effective batch of Alg. 1 (every gate open, every verification
// accepting the first or the second proposal): brute-force tree growth.  For
// depths with d1 | d2 and d1 | R it equals the branch-growth recurrence
// B = sum_k s_k, s_k = s_{k-1} + s_{k - d2/d1} (Sec. 4.3).
int worst_case_tree(int R, int d1, int d2, int accept) {
    struct N {
        int r, parent;
        std::vector<int> kids;
    };
    std::vector<N> nodes;
    std::vector<int> alive{0};
    nodes.push_back({0, -1, {}});
    int root = 0, peak = 1;
    for (int step = 0; step < 16 * R; ++step) {
        peak = std::max(peak, (int)alive.size());
        std::vector<int> cur = alive;
        for (int b : cur) {
            nodes[b].r += 1;
            if (nodes[b].r == d1 || (d2 && nodes[b].r == d2)) {
                nodes.push_back({0, b, {}});
                const int id = (int)nodes.size() - 1;
                nodes[b].kids.push_back(id);
                alive.push_back(id);
            }
        }
        if (nodes[root].r == R) {
            const auto& k = nodes[root].kids;
            const int keep = k[std::min<int>(accept, (int)k.size()) - 1];
            std::vector<int> next, stack{keep};
            while (!stack.empty()) {
                const int x = stack.back();
                stack.pop_back();
                next.push_back(x);
                for (int c : nodes[x].kids) stack.push_back(c);
            }
            std::vector<int> na;
            for (int x : alive)
                if (std::find(next.begin(), next.end(), x) != next.end()) na.push_back(x);
            alive = na;
            nodes[keep].parent = -1;
            root = keep;
        }
        peak = std::max(peak, (int)alive.size());
    }
    return peak;
}

}  // namespace

struct loopspec_handle {
    loopspec_dims d{};
    loopspec_config c{};
    hipStream_t st = nullptr;
    bool own_stream = false;
    bool bf16 = true;
    int wbytes = 2;
    Geo g{};
    int S = 0, worst = 0;
    int chunks_cap = 0;
    std::string err;

    // device buffers
    std::vector<void*> allocs;
    float *X = nullptr, *qbuf = nullptr, *logits = nullptr, *tmax = nullptr;
    PassBuf pb{};                 // row-ordered rounded state + sums of squares of the current pass
    std::vector<void*> folded;    // packed weight copies (owned)
    float *rope = nullptr;
    void *att = nullptr, *act = nullptr, *kvc = nullptr, *kvs = nullptr;
    int32_t *targ = nullptr;
    int32_t* mode = nullptr;
    // prefill rows: [R+1 depths][64] + coda copies [R][64] + LM-head row
    Row *pf_rows = nullptr, *pf_coda = nullptr, *pf_last = nullptr;
    int32_t *pf_n = nullptr, *pf_one = nullptr, *pf_jobs = nullptr;
    Sched sch{};
    int xrow_pf = 0, xrow_coda = 0, xrow_pf_coda = 0;

    // host staging (pinned)
    char* pin = nullptr;
    size_t pin_bytes = 0;

    // weights
    bool bound = false;
    const void *embed = nullptr, *final_norm = nullptr, *head = nullptr;
    std::vector<loopspec_layer_weights> layers;
    struct PackedLayer {
        const void *qkv = nullptr, *o = nullptr, *gu = nullptr, *down = nullptr;
    };
    std::vector<PackedLayer> packed;   // MFMA-order copies (owned, in `folded`)
    const void* head_packed = nullptr;

    // gemm configs: [0] direct path (<= 16 rows), [1] 64-row path
    GemmCfg cfg_qkv[2], cfg_o[2], cfg_gu[2], cfg_down[2], cfg_head[2];
    float* gpart = nullptr;       // split-k partials of the direct path
    unsigned* gcnt = nullptr;     // split-k arrival counters (one per tile, zero between launches)

    // persistent pass kernel (decode passes of <= 16 rows)
    bool pass_on = false;
    int pass_grid = 0;
    GemmCfg pcfg[4];              // qkv, o, gate/up, down
    int pitems[4] = {0, 0, 0, 0};
    const void** wl = nullptr;    // device: [L][4] packed weights per block
    unsigned* acnt = nullptr;     // device: attention counters of the pass kernel
    float* apart = nullptr;       // device: attention chunk partials of the pass kernel
    PassFlow flow{};              // device: per-block activation buffers of the pass kernel

    // graph
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
    hipGraph_t graph4 = nullptr;      // kStepsPerGraph steps back to back
    hipGraphExec_t exec4 = nullptr;
    int tree_mode = MODE_LOOPSPEC;
    float* skpart = nullptr;           // stream-K GEMM partials handed between waves (sentinel between launches)
    size_t skpart_n = 0;
    float* attn_part = nullptr;        // shared-prefix attention: partials of every (row, head)
    unsigned* attn_cnt = nullptr;      // ... and their counters (zero between launches)
    std::vector<int> prompt_len, first_tok, fresh;
    // coda models: coda_cov[q][r] = 1 while every committed position of
    // sequence q holds coda keys / values at depth r (a readout at depth r
    // attends to them).  The prefill writes every depth; a decode writes only
    // its readout depths for the positions it commits.
    std::vector<std::vector<uint8_t>> coda_cov;
    hipEvent_t ev0 = nullptr, ev1 = nullptr;
    float last_ms = 0.f;

    // measurement: HIP events around every launch of one kernel kind while a
    // profiled decode enqueues its steps directly (LOOPSPEC_PROF_* kinds; -1: off)
    int prof_kind = -1;
    std::vector<hipEvent_t> prof_ev;   // start / end pairs of the current step
    int prof_n = 0;                    // events recorded in the current step
};

namespace {

// event before / after a launch of the profiled kind (ignored when off or full)
// Arm the launch probe with the next event pair when this enqueue is the
// profiled kernel; prof_done keeps the pair only if a launch took it.
bool prof_arm(loopspec_t h, bool match) {
    if (!match || h->prof_kind < 0 || h->prof_n + 2 > (int)h->prof_ev.size()) return false;
    LaunchProbe& pr = launch_probe();
    pr.start = h->prof_ev[h->prof_n];
    pr.stop = h->prof_ev[h->prof_n + 1];
    pr.armed = true;
    return true;
}
void prof_done(loopspec_t h, bool armed) {
    if (!armed) return;
    LaunchProbe& pr = launch_probe();
    if (pr.armed)
        pr.armed = false;              // nothing was launched
    else
        h->prof_n += 2;
}

int fail(loopspec_t h, int code, const std::string& msg) {
    if (h) h->err = msg;
    return code;
}

#define HIPCHK(h, x)                                                                    \
    do {                                                                                \
        hipError_t e_ = (x);                                                            \
        if (e_ != hipSuccess)                                                           \
            return fail(h, LOOPSPEC_EHIP, std::string(#x) + ": " + hipGetErrorString(e_)); \
    } while (0)

template <typename T>
int dalloc(loopspec_t h, T** p, size_t n) {
    void* q = nullptr;
    if (hipMalloc(&q, std::max<size_t>(n, 1) * sizeof(T)) != hipSuccess) {
        (void)hipGetLastError();
        return fail(h, LOOPSPEC_ENOMEM, "device allocation of " + std::to_string(n * sizeof(T)) + " bytes failed");
    }
    h->allocs.push_back(q);
    *p = (T*)q;
    return LOOPSPEC_OK;
}

// Launch configuration of the standalone GEMM.  nt_max = 1: the direct path
// (at most 16 rows), where each wave holds all of its k steps in registers,
// at most gemm_max_steps(epi, 1) of them: k is cut into ks * kg contiguous
// slices, ks per workgroup and kg workgroups per tile.  nt_max > 1: the
// 64-row path, which streams k in rounds.  c.ok = false when no split fits.
GemmCfg pick_cfg(const loopspec_t h, int tiles, int K, int nmat, int epi, int nt_max) {
    GemmCfg c;
    const int kstep = h->bf16 ? 32 : 16;
    const int nsteps = K / kstep;
    const int vec = h->bf16 ? 8 : 4;
    if (nt_max <= 1) {
        const int per = gemm_max_steps(epi, 1);
        int KS = (nsteps + per - 1) / per;             // fewest slices whose shares fit
        const int want = (kWaveTarget + tiles - 1) / tiles;
        KS = std::max(KS, std::min(want, nsteps / 3)); // thin launches: more slices, >= 3 steps each
        int kg = (KS + 15) / 16;
        kg = std::max(kg, std::min(KS, (kWgTarget + tiles - 1) / tiles));
        kg = std::min(kg, 16);
        c.kg = kg;
        c.ks = (KS + kg - 1) / kg;
        if (c.ks > 16) c.ok = false;
        const int KSt = c.ks * c.kg;
        if ((nsteps + KSt - 1) / KSt > per) c.ok = false;
        if (c.kg == 1)
            while (c.tpw * c.ks < 8 && tiles / (c.tpw * 2) >= 512) c.tpw *= 2;
        c.kc = kstep;
        while (gemm_lds_bytes(h->wbytes, epi, nmat, c.tpw, c.ks, c.kc, 1, c.kg) > kLdsBudget && c.tpw > 1) c.tpw /= 2;
        if (gemm_lds_bytes(h->wbytes, epi, nmat, c.tpw, c.ks, c.kc, 1, c.kg) > kLdsMax) c.ok = false;
        return c;
    }
    // 64-row path: each wave streams its steps (every ks-th) in rounds
    const int per = gemm_max_steps(epi, 4);
    c.ks = std::min(16, std::max(1, (nsteps + per - 1) / per));
    // more slices while the launch has few waves (latency hiding), up to 16 per workgroup
    while (c.ks * 2 <= 16 && tiles * c.ks < 2048 && nsteps / (c.ks * 2) >= 2) c.ks *= 2;
    while (c.tpw * c.ks < 8 && tiles / (c.tpw * 2) >= 512) c.tpw *= 2;
    // LDS k chunk: the activation tile of nt_max*16 rows must fit the budget
    int kc = (int)(kLdsBudget - 256) / (nt_max * 16 * h->wbytes) - vec;
    kc = std::max(kstep, kc / kstep * kstep);
    c.kc = std::min(kc, K);
    while (gemm_lds_bytes(h->wbytes, epi, nmat, c.tpw, c.ks, c.kc, nt_max) > kLdsBudget && c.tpw > 1) c.tpw /= 2;
    if (gemm_lds_bytes(h->wbytes, epi, nmat, c.tpw, c.ks, c.kc, nt_max) > kLdsMax) c.ok = false;
    return c;
}

// Work split of one kind inside the persistent pass: 8 waves per workgroup as
// tpw tiles x ks k-slices, at most one work item per workgroup and at most
// pass_max_steps k steps per wave.  The smallest tpw that fits spreads the
// weight stream over the most CUs.
bool pick_pass_cfg(const loopspec_t h, int tiles, int K, int kind, int grid, GemmCfg* c, int* items) {
    const int nsteps = K / (h->bf16 ? 32 : 16);
    bool found = false;
    for (int tpw = 1; tpw <= kPassThreads / 64; tpw *= 2) {
        const int ks = kPassThreads / 64 / tpw;
        const int it = (tiles + tpw - 1) / tpw;
        if (it <= grid && (nsteps + ks - 1) / ks <= pass_max_steps(kind, h->g.h > 2048)) {
            c->tpw = tpw;
            c->ks = ks;
            c->kc = 32;
            *items = it;
            found = true;
            if (kind != PK_O) break;
        }
    }
    return found;
}

GemmParams gemm_base(loopspec_t h, const Row* rows, const int32_t* nrows) {
    GemmParams p{};
    p.g = h->g;
    p.kg = 1;
    p.part = h->gpart;
    p.cnt = h->gcnt;
    p.rows = rows;
    p.nrows = nrows;
    p.XB = h->pb.XB;
    p.SSQR = h->pb.SSQR;
    p.X = h->X;
    p.XBout = h->pb.XB;
    p.SSQRout = h->pb.SSQR;
    p.err = h->sch.err;
    return p;
}

hipError_t run_gemm(loopspec_t h, GemmParams p, int epi, const GemmCfg& c, int nt_max) {
    const int si = nt_max <= 1 ? 0 : nt_max <= 2 ? 1 : nt_max <= 4 ? 2 : -1;
    if (si >= 0 && c.sk_grid[si] > 0) {
        p.kg = c.sk_c[si];
        p.part = h->skpart;
        if (!p.err) p.err = h->sch.err;
        return launch_gemm_sk(p, epi, h->bf16, 1 << si, c.sk_grid[si], h->st);
    }
    p.ks = c.ks;
    p.tpw = c.tpw;
    p.kc = c.kc;
    p.kg = nt_max <= 1 ? c.kg : 1;
    return launch_gemm(p, epi, h->bf16, nt_max, h->st);
}

// One launch of kernel `k` (0 QKV, 1 attention, 2 O, 3 gate/up, 4 down) of
// block `l` of a stack over a row list.  big = prefill-sized row list.
hipError_t enqueue_kernel_(loopspec_t h, int k, int stack, int l, const Row* rows, const int32_t* nrows,
                           int rows_cap, bool big) {
    const int nt_max = (rows_cap + 15) / 16;
    const int first = stack == STACK_PRE ? 0 : stack == STACK_CORE ? h->g.Lp : h->g.Lp + h->g.Lb;
    const int hd = h->g.h, F = h->g.F;
    const int b = nt_max > 1 ? 1 : 0;            // direct path (<= 16 rows) or 64-row path
    (void)big;
    const loopspec_handle::PackedLayer& w = h->packed[first + l];
    hipError_t e = hipSuccess;
    switch (k) {
        case 0: {   // RMSNorm + QKV + RoPE + KV write
            GemmParams p = gemm_base(h, rows, nrows);
            p.K = hd;
            p.Wp = w.qkv;
            p.N_mat = hd;
            p.tiles = 3 * hd / kTile;
            p.qout = h->qbuf;
            p.kvc = h->kvc;
            p.kvs = h->kvs;
            p.rope = h->rope;
            p.stack = stack;
            p.layer = l;
            return run_gemm(h, p, EPI_QKV, h->cfg_qkv[b], nt_max);
        }
        case 1: {   // attention at each row's own depth
            AttnParams a{};
            a.g = h->g;
            a.nrows = nrows;
            a.rows = rows;
            a.q = h->qbuf;
            a.kvc = h->kvc;
            a.kvs = h->kvs;
            a.stack = stack;
            a.layer = l;
            a.chunks_cap = h->chunks_cap;
            a.out = h->att;
            const bool tasks = !big && h->attn_part;
            return launch_attention(a, h->bf16, rows_cap, tasks ? h->attn_part : nullptr, tasks ? h->attn_cnt : nullptr,
                                    h->st);
        }
        case 2: {   // O projection + residual
            GemmParams p = gemm_base(h, rows, nrows);
            p.abuf = h->att;
            p.K = hd;
            p.Wp = w.o;
            p.N_mat = hd;
            p.tiles = hd / kTile;
            return run_gemm(h, p, EPI_RESID, h->cfg_o[b], nt_max);
        }
        case 3: {   // RMSNorm + gate/up + SwiGLU
            GemmParams p = gemm_base(h, rows, nrows);
            p.K = hd;
            p.Wp = w.gu;
            p.N_mat = F;
            p.tiles = F / kTile;
            p.act = h->act;
            return run_gemm(h, p, EPI_SWIGLU, h->cfg_gu[b], nt_max);
        }
        case 4: {   // down projection + residual
            GemmParams p = gemm_base(h, rows, nrows);
            p.abuf = h->act;
            p.K = F;
            p.Wp = w.down;
            p.N_mat = hd;
            p.tiles = hd / kTile;
            return run_gemm(h, p, EPI_RESID, h->cfg_down[b], nt_max);
        }
    }
    return e;
}

hipError_t enqueue_kernel(loopspec_t h, int k, int stack, int l, const Row* rows, const int32_t* nrows,
                          int rows_cap, bool big) {
    const bool armed = prof_arm(h, stack == STACK_CORE && h->prof_kind == LOOPSPEC_PROF_QKV + k);
    const hipError_t e = enqueue_kernel_(h, k, stack, l, rows, nrows, rows_cap, big);
    prof_done(h, armed);
    return e;
}

// Parameters of the persistent pass of a block stack over a row list.
PassParams pass_params(loopspec_t h, int stack, const Row* rows, const int32_t* nrows) {
    const int first = stack == STACK_PRE ? 0 : stack == STACK_CORE ? h->g.Lp : h->g.Lp + h->g.Lb;
    const int hd = h->g.h, F = h->g.F;
    PassParams pp{};
    GemmParams* kinds[4] = {&pp.qkv, &pp.o, &pp.gu, &pp.down};
    for (int k = 0; k < 4; ++k) {
        *kinds[k] = gemm_base(h, rows, nrows);
        kinds[k]->tpw = h->pcfg[k].tpw;
        kinds[k]->ks = h->pcfg[k].ks;
        kinds[k]->kc = h->pcfg[k].kc;
    }
    pp.qkv.K = hd;
    pp.qkv.N_mat = hd;
    pp.qkv.tiles = 3 * hd / kTile;
    pp.qkv.qout = h->qbuf;
    pp.qkv.kvc = h->kvc;
    pp.qkv.kvs = h->kvs;
    pp.qkv.rope = h->rope;
    pp.qkv.stack = stack;
    pp.o.abuf = h->att;
    pp.o.K = hd;
    pp.o.N_mat = hd;
    pp.o.tiles = hd / kTile;
    pp.gu.K = hd;
    pp.gu.N_mat = F;
    pp.gu.tiles = F / kTile;
    pp.gu.act = h->act;
    pp.down.abuf = h->act;
    pp.down.K = F;
    pp.down.N_mat = hd;
    pp.down.tiles = hd / kTile;
    AttnParams& a = pp.attn;
    a.g = h->g;
    a.nrows = nrows;
    a.rows = rows;
    a.q = h->qbuf;
    a.kvc = h->kvc;
    a.kvs = h->kvs;
    a.stack = stack;
    a.chunks_cap = h->chunks_cap;
    a.out = h->att;
    pp.wl = h->wl + 4 * first;
    pp.L = stack == STACK_PRE ? h->g.Lp : stack == STACK_CORE ? h->g.Lb : h->g.Lc;
    pp.flow = h->flow;
    pp.stack = stack;
    pp.attn_wg = h->chunks_cap <= kPassAttnWgChunks;
    pp.acnt = h->acnt;
    pp.apart = h->apart;
    pp.err = h->sch.err;
    a.err = h->sch.err;
    pp.items_qkv = h->pitems[0];
    pp.items_o = h->pitems[1];
    pp.items_gu = h->pitems[2];
    pp.items_down = h->pitems[3];
    return pp;
}

// One pass of a block stack over a row list (starting from the rows' X): the
// preparation + persistent pass kernel for decode row lists when it is
// enabled, else the gather + five launches per block.
hipError_t enqueue_stack(loopspec_t h, int stack, const Row* rows, const int32_t* nrows, int rows_cap, bool big) {
    const int n = stack == STACK_PRE ? h->g.Lp : stack == STACK_CORE ? h->g.Lb : h->g.Lc;
    hipError_t e;
    if (!big && h->pass_on && rows_cap <= kPassRows) {
        const PassParams pp = pass_params(h, stack, rows, nrows);
        if ((e = launch_pass_prep(pp, h->bf16, rows_cap, h->st)) != hipSuccess) return e;
        const bool armed = prof_arm(h, stack == STACK_CORE && h->prof_kind == LOOPSPEC_PROF_PASS);
        e = launch_pass(pp, h->bf16, h->pass_grid, h->st);
        prof_done(h, armed);
        return e;
    }
    if ((e = launch_gather(h->g, rows, nrows, rows_cap, h->X, h->pb, h->bf16, h->st)) != hipSuccess) return e;
    for (int l = 0; l < n; ++l)
        for (int k = 0; k < 5; ++k) {
            e = enqueue_kernel(h, k, stack, l, rows, nrows, rows_cap, big);
            if (e != hipSuccess) return e;
        }
    return hipSuccess;
}

hipError_t enqueue_head(loopspec_t h, const Row* rows, const int32_t* nrows, int rows_cap) {
    hipError_t e = launch_gather(h->g, rows, nrows, rows_cap, h->X, h->pb, h->bf16, h->st);
    if (e != hipSuccess) return e;
    GemmParams p = gemm_base(h, rows, nrows);
    p.K = h->g.h;
    p.Wp = h->head_packed;
    p.N_mat = h->g.V;
    p.tiles = (h->g.V + kTile - 1) / kTile;
    p.logits = h->logits;
    p.tmax = h->tmax;
    p.targ = h->targ;
    const int nt_max = (rows_cap + 15) / 16;
    const bool armed = prof_arm(h, h->prof_kind == LOOPSPEC_PROF_HEAD);
    e = run_gemm(h, p, EPI_LOGITS, h->cfg_head[nt_max > 1 ? 1 : 0], nt_max);
    prof_done(h, armed);
    return e;
}

hipError_t enqueue_finalize(loopspec_t h, const Sched& s, int fin_op, int rows_cap) {
    const int tiles = (h->g.V + kTile - 1) / kTile;
    if (h->c.temperature == 0.f) return launch_finalize_greedy(s, fin_op, h->tmax, h->targ, tiles, rows_cap, h->st);
    return launch_finalize_sample(s, fin_op, h->logits, rows_cap, h->st);
}

// The whole decode step (captured once into a graph).
hipError_t enqueue_step(loopspec_t h) {
    Sched& s = h->sch;
    hipError_t e;
    if ((e = enqueue_stack(h, STACK_CORE, s.rowsB, s.nB, h->S, false)) != hipSuccess) return e;
    if (h->g.Lc) {
        if ((e = launch_copy_rows(h->g, s.rowsC, s.nC, h->S, h->X, h->st)) != hipSuccess) return e;
        if ((e = enqueue_stack(h, STACK_CODA, s.rowsC, s.nC, h->S, false)) != hipSuccess) return e;
    }
    if ((e = enqueue_head(h, s.rowsC, s.nC, h->S)) != hipSuccess) return e;
    if ((e = enqueue_finalize(h, s, FIN_STEP, h->S)) != hipSuccess) return e;
    if ((e = launch_sched(s, OP_STEP, 0, 0, nullptr, h->st)) != hipSuccess) return e;
    if ((e = launch_commit_embed(s, h->kvc, h->kvs, h->wbytes, h->embed, h->bf16, h->X, h->st)) != hipSuccess)
        return e;
    if (h->g.Lp) {
        if ((e = enqueue_stack(h, STACK_PRE, s.rowsP, s.nP, h->S, false)) != hipSuccess) return e;
    }
    return hipSuccess;
}

// One decode step captured as a graph, and kStepsPerGraph steps in one more
// graph: consecutive replays of a graph leave a gap of several microseconds
// between them on the GPU, so long decodes replay the multi-step graph.
constexpr int kStepsPerGraph = 4;

static int capture_steps(loopspec_t h, int steps, hipGraph_t* graph, hipGraphExec_t* exec) {
    HIPCHK(h, hipStreamBeginCapture(h->st, hipStreamCaptureModeThreadLocal));
    hipError_t e = hipSuccess;
    for (int i = 0; i < steps && e == hipSuccess; ++i) e = enqueue_step(h);
    hipGraph_t g = nullptr;
    hipError_t e2 = hipStreamEndCapture(h->st, &g);
    if (e != hipSuccess) return fail(h, LOOPSPEC_EHIP, std::string("step capture: ") + hipGetErrorString(e));
    if (e2 != hipSuccess) return fail(h, LOOPSPEC_EHIP, std::string("end capture: ") + hipGetErrorString(e2));
    *graph = g;
    HIPCHK(h, hipGraphInstantiate(exec, g, nullptr, nullptr, 0));
    return LOOPSPEC_OK;
}

// the step graphs carry the scheduler's settings in their kernel arguments:
// dropped whenever those change, captured again by the next decode call
void drop_graphs(loopspec_t h) {
    if (h->exec) (void)hipGraphExecDestroy(h->exec);
    if (h->graph) (void)hipGraphDestroy(h->graph);
    if (h->exec4) (void)hipGraphExecDestroy(h->exec4);
    if (h->graph4) (void)hipGraphDestroy(h->graph4);
    h->exec = h->exec4 = nullptr;
    h->graph = h->graph4 = nullptr;
}

int ensure_graph(loopspec_t h) {
    if (h->exec) return LOOPSPEC_OK;
    int r = capture_steps(h, 1, &h->graph, &h->exec);
    if (r) return r;
    return capture_steps(h, kStepsPerGraph, &h->graph4, &h->exec4);
}

int check_err(loopspec_t h) {
    int32_t e = 0;
    HIPCHK(h, hipMemcpyAsync(&e, h->sch.err, 4, hipMemcpyDeviceToHost, h->st));
    HIPCHK(h, hipStreamSynchronize(h->st));
    if (e & ERR_NUMERIC) return fail(h, LOOPSPEC_ENUMERIC, "NaN/Inf in readout logits");
    if (e & ERR_CTX) return fail(h, LOOPSPEC_ECAPACITY, "context capacity reached during decoding");
    if (e & ERR_SLOTS) return fail(h, LOOPSPEC_ECAPACITY, "no free branch slot");
    if (e & ERR_TREE) return fail(h, LOOPSPEC_ESTATE, "inconsistent branch tree: a decision without its first draft");
    if (e & ERR_SYNC) {
        // a wait inside a launch gave up: reset the sampler's barrier state so the
        // handle stays usable
        if (h->sch.srow)
            HIPCHK(h, hipMemsetAsync(h->sch.srow, 0, (size_t)h->S * kRowWords * 8, h->st));
        if (h->skpart) HIPCHK(h, hipMemsetAsync(h->skpart, 0xFF, h->skpart_n * 4, h->st));
        HIPCHK(h, hipStreamSynchronize(h->st));
        return fail(h, LOOPSPEC_EHIP, "a wait inside a launch gave up (pass kernel data or sampler shards)");
    }
    return LOOPSPEC_OK;
}

int set_mode(loopspec_t h, int mode) {
    HIPCHK(h, hipMemcpyAsync(h->mode, &mode, 4, hipMemcpyHostToDevice, h->st));
    HIPCHK(h, hipStreamSynchronize(h->st));
    return LOOPSPEC_OK;
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================
extern "C" {

const char* loopspec_version(void) { return "loopspec-gfx950 0.1"; }

int32_t loopspec_worst_case_branches(int32_t R, int32_t d1, int32_t d2) {
    if (R < 2 || d1 < 1 || d1 >= R || (d2 != 0 && !(d1 < d2 && d2 < R)) || R / d1 >= kChainMax) return -1;
    return std::max(worst_case_tree(R, d1, d2, 1), worst_case_tree(R, d1, d2, 2));
}

const char* loopspec_last_error(loopspec_t h) { return h ? h->err.c_str() : "null handle"; }

void loopspec_destroy(loopspec_t h) {
    if (!h) return;
    if (h->st) (void)hipStreamSynchronize(h->st);
    drop_graphs(h);
    if (h->ev0) (void)hipEventDestroy(h->ev0);
    if (h->ev1) (void)hipEventDestroy(h->ev1);
    for (hipEvent_t e : h->prof_ev) (void)hipEventDestroy(e);
    for (void* p : h->allocs) (void)hipFree(p);
    if (h->pin) (void)hipHostFree(h->pin);
    for (void* p : h->folded) (void)hipFree(p);
    if (h->own_stream && h->st) (void)hipStreamDestroy(h->st);
    delete h;
}

int loopspec_create(const loopspec_dims* dims, const loopspec_config* cfg, void* stream, loopspec_t* out) {
    if (!dims || !cfg || !out) return LOOPSPEC_EINVAL;
    *out = nullptr;
    loopspec_t h = new loopspec_handle();
    h->d = *dims;
    h->c = *cfg;
    h->st = (hipStream_t)stream;
    const loopspec_dims& d = h->d;
    const loopspec_config& c = h->c;
    auto bad = [&](const std::string& m) {
        const int r = fail(h, LOOPSPEC_EINVAL, m);
        *out = h;
        return r;
    };
    if (d.hidden <= 0 || d.n_heads <= 0 || d.head_dim <= 0 || d.ffn <= 0 || d.vocab <= 0)
        return bad("dimensions must be positive");
    if (d.hidden != d.n_heads * d.head_dim) return bad("hidden must equal n_heads * head_dim");
    if (d.head_dim != 16 && d.head_dim != 32 && d.head_dim != 64 && d.head_dim != 96 && d.head_dim != 128)
        return bad("head_dim must be 16, 32, 64, 96 or 128");
    if (d.weight_dtype == LOOPSPEC_F32 && d.head_dim > 64) return bad("fp32 models need head_dim <= 64");
    if (d.hidden % 32 || d.ffn % 32) return bad("hidden and ffn must be multiples of 32");
    if (d.n_core <= 0 || d.n_prelude < 0 || d.n_coda < 0) return bad("need n_core > 0, n_prelude, n_coda >= 0");
    if (d.weight_dtype != LOOPSPEC_F32 && d.weight_dtype != LOOPSPEC_BF16) return bad("unknown weight_dtype");
    if (d.max_seqs <= 0 || d.max_ctx < 4) return bad("max_seqs > 0 and max_ctx >= 4 required");
    if (!(d.rms_eps > 0.f) || !(d.rope_base > 0.f)) return bad("rms_eps and rope_base must be positive");
    if (c.R < 2 || c.d1 < 1 || c.d1 >= c.R) return bad("need 1 <= d1 < R");
    if (c.d2 != 0 && !(c.d1 < c.d2 && c.d2 < c.R)) return bad("need d1 < d2 < R, or d2 = 0");
    if (c.temperature < 0.f || !(c.top_p > 0.f && c.top_p <= 1.f)) return bad("need temperature >= 0, 0 < top_p <= 1");
    if (c.max_slots < 0) return bad("max_slots must be >= 0");
    if (c.shared_prefix != 0 && c.shared_prefix != 1) return bad("shared_prefix must be 0 or 1");
    if (c.temperature > 0.f && d.vocab > kSampleMaxVocab)
        return bad("sampling supports vocabularies up to " + std::to_string(kSampleMaxVocab));
    if (c.second_proposal < LOOPSPEC_SP_GATED || c.second_proposal > LOOPSPEC_SP_NAIVE)
        return bad("unknown second_proposal variant");
    if (c.second_proposal != LOOPSPEC_SP_GATED && (c.temperature == 0.f || c.d2 == 0))
        return bad("the ungated second-proposal variants need temperature > 0 and d2 > 0");
    if (c.R / c.d1 >= kChainMax) return bad("R / d1 must be below " + std::to_string(kChainMax));

    h->bf16 = d.weight_dtype == LOOPSPEC_BF16;
    h->wbytes = h->bf16 ? 2 : 4;
    h->worst = std::max(worst_case_tree(c.R, c.d1, c.d2, 1), worst_case_tree(c.R, c.d1, c.d2, 2));
    h->S = c.max_slots ? c.max_slots : h->worst * d.max_seqs;
    if (h->S < d.max_seqs) h->S = d.max_seqs;
    if (h->S > kMaxRows) {
        const int r = fail(h, LOOPSPEC_ECAPACITY,
                           "branch slots " + std::to_string(h->S) + " exceed the 64 rows of one batched pass");
        *out = h;
        return r;
    }
    Geo& g = h->g;
    g.h = d.hidden;
    g.H = d.n_heads;
    g.dh = d.head_dim;
    g.F = d.ffn;
    g.V = d.vocab;
    g.Lp = d.n_prelude;
    g.Lb = d.n_core;
    g.Lc = d.n_coda;
    g.R = c.R;
    g.T = g.Lp + c.R * g.Lb + c.R * g.Lc;
    g.max_ctx = d.max_ctx;
    g.S = h->S;
    g.ssq_tiles = d.hidden / 16;
    g.eps = d.rms_eps;
    g.attn_scale = (float)(1.0 / std::sqrt((double)d.head_dim));
    h->chunks_cap = (d.max_ctx + kChunk - 1) / kChunk;
    *out = h;

    // a graph cannot be captured on the legacy default stream: use our own
    if (!h->st) {
        HIPCHK(h, hipStreamCreateWithFlags(&h->st, hipStreamNonBlocking));
        h->own_stream = true;
    }
    HIPCHK(h, gemm_prepare((int)kLdsMax));
    const int S = h->S;
    const int xrows = S + kPrefillRows + std::max(S, kPrefillRows);
    h->xrow_pf = S;
    h->xrow_coda = S + kPrefillRows;
    h->xrow_pf_coda = S + kPrefillRows;
    const int rmax = std::max(S, kPrefillRows);
    const size_t V = d.vocab, tiles = (V + 15) / 16;
    int r;
    if ((r = dalloc(h, &h->X, (size_t)xrows * g.h))) return r;
    if ((r = dalloc(h, (char**)&h->pb.XB, (size_t)kMaxRows * g.h * h->wbytes))) return r;
    if ((r = dalloc(h, &h->pb.SSQR, (size_t)kMaxRows * g.ssq_tiles))) return r;
    if ((r = dalloc(h, &h->qbuf, (size_t)rmax * g.h))) return r;
    if ((r = dalloc(h, (char**)&h->att, (size_t)rmax * g.h * h->wbytes))) return r;
    if ((r = dalloc(h, (char**)&h->act, (size_t)rmax * g.F * h->wbytes))) return r;
    {
        const size_t lds = attention_lds_bytes(h->chunks_cap, g.dh);
        if (lds > 160 * 1024) return fail(h, LOOPSPEC_ECAPACITY, "max_ctx too large for the attention workgroup's LDS");
        HIPCHK(h, attention_prepare((int)lds));
    }
    if (c.shared_prefix) {
        if ((r = dalloc(h, &h->attn_part, attention_partials_floats(S, g.H, h->chunks_cap, g.dh)))) return r;
        if ((r = dalloc(h, &h->attn_cnt, (size_t)S * g.H))) return r;
        HIPCHK(h, hipMemset(h->attn_cnt, 0, (size_t)S * g.H * sizeof(unsigned)));
    }
    if ((r = dalloc(h, &h->logits, (size_t)S * V))) return r;
    if ((r = dalloc(h, &h->tmax, (size_t)S * tiles))) return r;
    if ((r = dalloc(h, &h->targ, (size_t)S * tiles))) return r;
    if ((r = dalloc(h, (char**)&h->kvc, (size_t)d.max_seqs * g.T * 2 * d.max_ctx * g.h * h->wbytes))) return r;
    if ((r = dalloc(h, (char**)&h->kvs, (size_t)S * g.T * 2 * g.h * h->wbytes))) return r;
    if ((r = dalloc(h, &h->rope, (size_t)d.max_ctx * g.dh))) return r;
    if ((r = dalloc(h, &h->mode, 1))) return r;
    if ((r = dalloc(h, &h->pf_rows, (size_t)(c.R + 1) * kPrefillRows))) return r;
    if ((r = dalloc(h, &h->pf_coda, (size_t)(c.R + 1) * kPrefillRows))) return r;
    if ((r = dalloc(h, &h->pf_last, 1))) return r;
    if ((r = dalloc(h, &h->pf_n, 2))) return r;
    h->pf_one = h->pf_n + 1;
    if ((r = dalloc(h, &h->pf_jobs, 2 * kPrefillRows))) return r;

    // scheduler tables
    Sched& s = h->sch;
    s.g = g;
    s.max_seqs = d.max_seqs;
    s.R = c.R;
    s.d1 = c.d1;
    s.d2 = c.d2;
    s.variant = c.second_proposal;
    s.greedy = c.temperature == 0.f;
    s.temperature = c.temperature;
    s.top_p = c.top_p;
    {
        unsigned long long* sd = nullptr;
        if ((r = dalloc(h, &sd, 1))) return r;
        HIPCHK(h, hipMemcpy(sd, &c.seed, 8, hipMemcpyHostToDevice));
        s.seed = sd;
    }
    s.mode = h->mode;
    int32_t** slot_tabs[] = {&s.s_active, &s.s_seq, &s.s_pos, &s.s_tok, &s.s_depth, &s.s_parent,
                             &s.s_c1, &s.s_c2, &s.s_x1, &s.s_x2, &s.s_gate};
    for (auto pp : slot_tabs)
        if ((r = dalloc(h, pp, S))) return r;
    int32_t** seq_tabs[] = {&s.q_root, &s.q_tdone, &s.q_ncommit, &s.q_target, &s.q_state, &s.q_last_tok,
                            &s.q_last_src};
    for (auto pp : seq_tabs)
        if ((r = dalloc(h, pp, d.max_seqs))) return r;
    if ((r = dalloc(h, &s.Y, (size_t)d.max_seqs * d.max_ctx))) return r;
    if ((r = dalloc(h, &s.forced, (size_t)d.max_seqs * d.max_ctx))) return r;
    if ((r = dalloc(h, &s.rowsB, S))) return r;
    if ((r = dalloc(h, &s.rowsC, S))) return r;
    if ((r = dalloc(h, &s.rowsP, S))) return r;
    if ((r = dalloc(h, &s.nB, 8))) return r;
    s.nC = s.nB + 1;
    s.nP = s.nB + 2;
    s.njc = s.nB + 3;
    s.njs = s.nB + 4;
    s.err = s.nB + 5;
    s.coda_xrow0 = g.Lc ? h->xrow_coda : -1;
    if ((r = dalloc(h, &s.ro_tok, S))) return r;
    if ((r = dalloc(h, &s.ro_aux, S))) return r;
    if ((r = dalloc(h, &s.jc, 3 * d.max_seqs))) return r;
    if ((r = dalloc(h, &s.js, 2 * S))) return r;
    if ((r = dalloc(h, &s.stats, ST_N))) return r;
    if (c.temperature > 0.f) {
        if ((r = dalloc(h, &s.q1, (size_t)S * V))) return r;
        if ((r = dalloc(h, &s.q2, (size_t)S * V))) return r;
        if ((r = dalloc(h, &s.q2t, (size_t)S * V))) return r;
        if (sample_rows_resident(d.vocab) < S)
            return fail(h, LOOPSPEC_ECAPACITY, "the sampling readout's shards of " + std::to_string(S) +
                                                   " rows do not fit on the GPU at once");
        if ((r = dalloc(h, &s.srow, (size_t)S * kRowWords))) return r;
        HIPCHK(h, hipMemsetAsync(s.srow, 0, (size_t)S * kRowWords * 8, h->st));
    }

    // zero the tables (outside any graph)
    HIPCHK(h, hipMemsetAsync(s.s_active, 0, S * 4, h->st));
    HIPCHK(h, hipMemsetAsync(s.s_seq, 0xFF, S * 4, h->st));
    HIPCHK(h, hipMemsetAsync(s.q_state, 0, d.max_seqs * 4, h->st));
    HIPCHK(h, hipMemsetAsync(s.nB, 0, 8 * 4, h->st));
    HIPCHK(h, hipMemsetAsync(s.stats, 0, ST_N * 8, h->st));
    HIPCHK(h, hipMemsetAsync(s.forced, 0, (size_t)d.max_seqs * d.max_ctx * 4, h->st));
    HIPCHK(h, hipMemsetAsync(h->mode, 0, 4, h->st));
    HIPCHK(h, hipMemsetAsync(h->X, 0, (size_t)xrows * g.h * 4, h->st));

    // RoPE table from fp64: angle = pos * base^(-2i/dh)
    {
        std::vector<float> t((size_t)d.max_ctx * g.dh);
        const int half = g.dh / 2;
        for (int p = 0; p < d.max_ctx; ++p)
            for (int i = 0; i < half; ++i) {
                const double a = (double)p * std::pow((double)d.rope_base, -2.0 * i / g.dh);
                t[((size_t)p * half + i) * 2] = (float)std::cos(a);
                t[((size_t)p * half + i) * 2 + 1] = (float)std::sin(a);
            }
        HIPCHK(h, hipMemcpy(h->rope, t.data(), t.size() * 4, hipMemcpyHostToDevice));
    }

    // launch configurations: the direct path (rows <= 16) and the 64-row path
    // (decode with more than 16 slots, prefill)
    {
        size_t part_elems = 0, sk_elems = 0;
        int cnt_n = 0;
        for (int b = 0; b < 2; ++b) {
            const int nt = b ? (kPrefillRows + 15) / 16 : 1;
            struct K { GemmCfg* c; int tiles, K, nmat, epi; } ks[] = {
                {&h->cfg_qkv[b], 3 * g.h / 16, g.h, 1, EPI_QKV}, {&h->cfg_o[b], g.h / 16, g.h, 1, EPI_RESID},
                {&h->cfg_gu[b], g.F / 16, g.h, 2, EPI_SWIGLU}, {&h->cfg_down[b], g.h / 16, g.F, 1, EPI_RESID},
                {&h->cfg_head[b], (int)tiles, g.h, 1, EPI_LOGITS}};
            for (const K& k : ks) {
                *k.c = pick_cfg(h, k.tiles, k.K, k.nmat, k.epi, nt);
                if (!k.c->ok)
                    return fail(h, LOOPSPEC_EINVAL, "no GEMM launch configuration fits K = " + std::to_string(k.K) +
                                                        " (registers of one wave, LDS of one CU)");
                if (k.c->kg > 1) {
                    part_elems = std::max(part_elems, (size_t)k.tiles * k.c->kg * k.nmat * 256);
                    cnt_n = std::max(cnt_n, k.tiles);
                }
                // launches of at most 16 rows stream the weights stream-K; wider
                // ones too when the launch streams at least kSkWideBytes (below
                // that, the stream-K fix-up and per-launch set-up cost more than
                // the 64-row tiles lose)
                const bool wide_sk = (size_t)k.tiles * 16 * k.K * h->wbytes * k.nmat >= kSkWideBytes;
                for (int si = b ? 1 : 0; si < (b ? (wide_sk ? 3 : 1) : 1); ++si) {
                    HIPCHK(h, gemm_sk_shape(k.epi, h->bf16, 1 << si, k.tiles, k.K, &k.c->sk_grid[si], &k.c->sk_c[si]));
                    sk_elems = std::max(sk_elems, (size_t)k.tiles * k.c->sk_c[si] * k.nmat * 256 * (1 << si));
                }
            }
        }
        if ((r = dalloc(h, &h->gpart, std::max<size_t>(part_elems, 1)))) return r;
        // stream-K hand-over slots hold the sentinel between launches
        h->skpart_n = std::max<size_t>(sk_elems, 1);
        if ((r = dalloc(h, &h->skpart, h->skpart_n))) return r;
        HIPCHK(h, hipMemsetAsync(h->skpart, 0xFF, h->skpart_n * 4, h->st));
        if ((r = dalloc(h, &h->gcnt, (size_t)std::max(cnt_n, 1)))) return r;
        HIPCHK(h, hipMemsetAsync(h->gcnt, 0, (size_t)std::max(cnt_n, 1) * 4, h->st));
    }
    // (decode and prefill may slice k differently: prefill only fills the
    // committed cache, which vanilla and LoopSpec decoding then share)

    // persistent pass: one 8-wave workgroup per CU, all co-resident
    {
        const int L = g.Lp + g.Lb + g.Lc;
        if ((r = dalloc(h, &h->wl, (size_t)4 * L))) return r;
        int dev = 0, cus = 0;
        HIPCHK(h, hipGetDevice(&dev));
        HIPCHK(h, hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
        const int G = cus;
        bool ok = !c.per_kernel && S <= kPassRows && G > 0 && h->chunks_cap <= 128;
        ok = ok && pick_pass_cfg(h, 3 * g.h / 16, g.h, PK_QKV, G, &h->pcfg[0], &h->pitems[0]);
        ok = ok && pick_pass_cfg(h, g.h / 16, g.h, PK_O, G, &h->pcfg[1], &h->pitems[1]);
        ok = ok && pick_pass_cfg(h, g.F / 16, g.h, PK_GU, G, &h->pcfg[2], &h->pitems[2]);
        ok = ok && pick_pass_cfg(h, g.h / 16, g.F, PK_DOWN, G, &h->pcfg[3], &h->pitems[3]);
        if (ok) {
            const int Lmax = std::max(g.Lb, std::max(g.Lp, g.Lc));
            char* fb = nullptr;
            // attention partials handed between workgroups: chunk tasks (long
            // contexts) or the parts of a row with more partials than waves
            if ((r = dalloc(h, &h->apart, (size_t)kPassRows * g.H * (h->chunks_cap + 1) * (g.dh + 2)))) return r;
            if ((r = dalloc(h, &h->acnt, (size_t)kPassRows * g.H))) return r;
            if ((r = dalloc(h, &fb, pass_flow_bytes(g, Lmax, h->wbytes)))) return r;
            h->flow = pass_flow_carve(fb, g, Lmax, h->wbytes);
        }
        if (ok) {
            PassParams pp = pass_params(h, STACK_CORE, nullptr, nullptr);
            const size_t lds = pass_lds_bytes(pp, h->wbytes);
            ok = lds <= 160 * 1024 && pass_prepare((int)lds, h->bf16, g.dh, g.h > 2048) == hipSuccess &&
                 pass_occupancy(h->bf16, g.dh, g.h > 2048, (int)lds) >= 1;
        }
        h->pass_on = ok;
        h->pass_grid = G;
    }

    h->pin_bytes = std::max<size_t>((size_t)(c.R + 1) * kPrefillRows * sizeof(Row) * 2 + 4096,
                                    (size_t)d.max_seqs * d.max_ctx * 4 + 4096);
    HIPCHK(h, hipHostMalloc((void**)&h->pin, h->pin_bytes, hipHostMallocDefault));
    HIPCHK(h, hipEventCreate(&h->ev0));
    HIPCHK(h, hipEventCreate(&h->ev1));
    h->prompt_len.assign(d.max_seqs, 0);
    h->first_tok.assign(d.max_seqs, -1);
    h->fresh.assign(d.max_seqs, 0);
    h->coda_cov.assign(d.max_seqs, std::vector<uint8_t>(c.R + 1, 1));
    HIPCHK(h, hipStreamSynchronize(h->st));
    return LOOPSPEC_OK;
}

int loopspec_bind_weights(loopspec_t h, const loopspec_weights* w) {
    if (!h) return LOOPSPEC_EINVAL;
    if (!w || !w->embed || !w->final_norm || !w->layers) return fail(h, LOOPSPEC_EINVAL, "null weight pointer");
    const int L = h->d.n_prelude + h->d.n_core + h->d.n_coda;
    if (w->n_layers != L) return fail(h, LOOPSPEC_EINVAL, "n_layers must be n_prelude + n_core + n_coda");
    if (!h->d.tied_head && !w->head) return fail(h, LOOPSPEC_EINVAL, "untied model needs a head matrix");
    for (int l = 0; l < L; ++l) {
        const loopspec_layer_weights& x = w->layers[l];
        const void* ps[] = {x.attn_norm, x.wq, x.wk, x.wv, x.wo, x.ffn_norm, x.wg, x.wu, x.wd};
        for (const void* p : ps)
            if (!p) return fail(h, LOOPSPEC_EINVAL, "null pointer in layer " + std::to_string(l));
    }
    h->embed = w->embed;
    h->final_norm = w->final_norm;
    h->head = h->d.tied_head ? w->embed : w->head;
    h->layers.assign(w->layers, w->layers + L);
    // pack every matrix into MFMA operand order, folding in the RMSNorm gain of
    // the matrices that read the normalised state
    for (void* p : h->folded) (void)hipFree(p);
    h->folded.clear();
    const int hd = h->d.hidden, F = h->d.ffn;
    auto pack = [&](int epi, const void* w0, const void* w1, const void* w2, const void* gain, int N, int K,
                    const void** out) -> int {
        const size_t bytes = packed_elems(epi, N, K, h->bf16) * h->wbytes;
        void* buf = nullptr;
        if (hipMalloc(&buf, bytes) != hipSuccess) {
            (void)hipGetLastError();
            return fail(h, LOOPSPEC_ENOMEM, "packed weight allocation failed");
        }
        h->folded.push_back(buf);
        const void* W[3] = {w0, w1, w2};
        hipError_t e = launch_pack(epi, W, gain, buf, N, K, h->g, h->bf16, h->sch.err, h->st);
        if (e != hipSuccess) return fail(h, LOOPSPEC_EHIP, hipGetErrorString(e));
        *out = buf;
        return LOOPSPEC_OK;
    };
    h->packed.assign(L, loopspec_handle::PackedLayer{});
    int r;
    {
        int32_t zero = 0;
        HIPCHK(h, hipMemcpyAsync(h->sch.err, &zero, 4, hipMemcpyHostToDevice, h->st));
    }
    for (int l = 0; l < L; ++l) {
        const loopspec_layer_weights& x = h->layers[l];
        loopspec_handle::PackedLayer& pk = h->packed[l];
        if ((r = pack(EPI_QKV, x.wq, x.wk, x.wv, x.attn_norm, hd, hd, &pk.qkv)) ||
            (r = pack(EPI_RESID, x.wo, nullptr, nullptr, nullptr, hd, hd, &pk.o)) ||
            (r = pack(EPI_SWIGLU, x.wg, x.wu, nullptr, x.ffn_norm, F, hd, &pk.gu)) ||
            (r = pack(EPI_RESID, x.wd, nullptr, nullptr, nullptr, hd, F, &pk.down)))
            return r;
    }
    if ((r = pack(EPI_LOGITS, h->head, nullptr, nullptr, h->final_norm, h->d.vocab, hd, &h->head_packed))) return r;
    {
        std::vector<const void*> wl((size_t)4 * L);
        for (int l = 0; l < L; ++l) {
            wl[4 * l] = h->packed[l].qkv;
            wl[4 * l + 1] = h->packed[l].o;
            wl[4 * l + 2] = h->packed[l].gu;
            wl[4 * l + 3] = h->packed[l].down;
        }
        HIPCHK(h, hipMemcpyAsync(h->wl, wl.data(), wl.size() * sizeof(void*), hipMemcpyHostToDevice, h->st));
    }
    HIPCHK(h, hipStreamSynchronize(h->st));
    {
        int32_t e = 0;
        HIPCHK(h, hipMemcpy(&e, h->sch.err, 4, hipMemcpyDeviceToHost));
        if (e & 1) return fail(h, LOOPSPEC_EINVAL, "a weight (times its RMSNorm gain) lies outside the fp16 range");
    }
    drop_graphs(h);
    h->bound = true;
    return LOOPSPEC_OK;
}

static int init_seq(loopspec_t h, int seq, int n, const int32_t* tok_dev) {
    Sched& s = h->sch;
    hipError_t e;
    if ((e = launch_sched(s, OP_INIT, seq, n, tok_dev, h->st)) != hipSuccess)
        return fail(h, LOOPSPEC_EHIP, hipGetErrorString(e));
    if ((e = launch_embed(h->g, s.js, s.njs, 1, h->embed, h->bf16, h->X, h->st)) != hipSuccess)
        return fail(h, LOOPSPEC_EHIP, hipGetErrorString(e));
    if (h->g.Lp && (e = enqueue_stack(h, STACK_PRE, s.rowsP, s.nP, h->S, false)) != hipSuccess)
        return fail(h, LOOPSPEC_EHIP, hipGetErrorString(e));
    h->fresh[seq] = 1;
    // the prompt (prefill) or the forced positions (every depth is a readout)
    std::fill(h->coda_cov[seq].begin(), h->coda_cov[seq].end(), 1);
    return LOOPSPEC_OK;
}

int loopspec_prefill(loopspec_t h, int32_t seq, const int32_t* ids, int32_t n, int32_t* first_tok) {
    if (!h) return LOOPSPEC_EINVAL;
    if (!h->bound) return fail(h, LOOPSPEC_ESTATE, "weights are not bound");
    if (seq < 0 || seq >= h->d.max_seqs) return fail(h, LOOPSPEC_EINVAL, "seq out of range");
    if (!ids || n < 1) return fail(h, LOOPSPEC_EINVAL, "empty prompt");
    if (n + 2 > h->d.max_ctx) return fail(h, LOOPSPEC_ECAPACITY, "prompt does not fit max_ctx");
    for (int i = 0; i < n; ++i)
        if (ids[i] < 0 || ids[i] >= h->d.vocab) return fail(h, LOOPSPEC_EINVAL, "token id out of range");
    const int R = h->c.R;
    const int Lc = h->g.Lc;
    Sched& s = h->sch;
    hipError_t e;
    int32_t zero = 0;
    HIPCHK(h, hipMemcpyAsync(s.err, &zero, 4, hipMemcpyHostToDevice, h->st));
    for (int p0 = 0; p0 < n; p0 += kPrefillRows) {
        const int m = std::min(kPrefillRows, n - p0);
        HIPCHK(h, hipStreamSynchronize(h->st));                 // staging buffer is free
        Row* rows = (Row*)h->pin;
        Row* coda = rows + (R + 1) * kPrefillRows;
        int32_t* misc = (int32_t*)(coda + (R + 1) * kPrefillRows);
        for (int r = 0; r <= R; ++r)
            for (int i = 0; i < m; ++i) {
                Row x{};
                x.xrow = h->xrow_pf + i;
                x.slot = -1;
                x.seq = seq;
                x.pos = p0 + i;
                x.depth = r;
                x.tdone = p0 + i;
                x.src = x.xrow;
                rows[r * kPrefillRows + i] = x;
                x.xrow = h->xrow_pf_coda + i;
                coda[r * kPrefillRows + i] = x;
            }
        misc[0] = m;
        misc[1] = 1;
        for (int i = 0; i < m; ++i) {
            misc[2 + 2 * i] = h->xrow_pf + i;
            misc[3 + 2 * i] = ids[p0 + i];
        }
        HIPCHK(h, hipMemcpyAsync(h->pf_rows, rows, sizeof(Row) * (R + 1) * kPrefillRows, hipMemcpyHostToDevice, h->st));
        HIPCHK(h, hipMemcpyAsync(h->pf_coda, coda, sizeof(Row) * (R + 1) * kPrefillRows, hipMemcpyHostToDevice, h->st));
        HIPCHK(h, hipMemcpyAsync(h->pf_n, misc, 8, hipMemcpyHostToDevice, h->st));
        HIPCHK(h, hipMemcpyAsync(h->pf_jobs, misc + 2, 8 * m, hipMemcpyHostToDevice, h->st));
        if ((e = launch_embed(h->g, h->pf_jobs, h->pf_n, m, h->embed, h->bf16, h->X, h->st)) != hipSuccess)
            return fail(h, LOOPSPEC_EHIP, hipGetErrorString(e));
        if (h->g.Lp && (e = enqueue_stack(h, STACK_PRE, h->pf_rows, h->pf_n, kPrefillRows, true)) != hipSuccess)
            return fail(h, LOOPSPEC_EHIP, hipGetErrorString(e));
        for (int r = 1; r <= R; ++r) {
            const Row* rr = h->pf_rows + r * kPrefillRows;
            if ((e = enqueue_stack(h, STACK_CORE, rr, h->pf_n, kPrefillRows, true)) != hipSuccess)
                return fail(h, LOOPSPEC_EHIP, hipGetErrorString(e));
            // coda caches of every readout depth (they are read by later readouts)
            if (Lc) {
                const Row* cr = h->pf_coda + r * kPrefillRows;
                if ((e = launch_copy_rows(h->g, cr, h->pf_n, kPrefillRows, h->X, h->st)) != hipSuccess)
                    return fail(h, LOOPSPEC_EHIP, hipGetErrorString(e));
                if ((e = enqueue_stack(h, STACK_CODA, cr, h->pf_n, kPrefillRows, true)) != hipSuccess)
                    return fail(h, LOOPSPEC_EHIP, hipGetErrorString(e));
            }
        }
        if (p0 + m == n) {
            // readout of the last prompt position at depth R
            Row last = (Lc ? coda : rows)[R * kPrefillRows + m - 1];
            HIPCHK(h, hipMemcpyAsync(h->pf_last, &last, sizeof(Row), hipMemcpyHostToDevice, h->st));
            if ((e = enqueue_head(h, h->pf_last, h->pf_one, 1)) != hipSuccess)
                return fail(h, LOOPSPEC_EHIP, hipGetErrorString(e));
            Sched t = s;
            t.rowsC = h->pf_last;
            t.nC = h->pf_one;
            if ((e = enqueue_finalize(h, t, FIN_TARGET, 1)) != hipSuccess)
                return fail(h, LOOPSPEC_EHIP, hipGetErrorString(e));
        }
    }
    // the prompt's ids at positions 0..n-1 of the sequence's token record
    // (committed tokens follow them), for loopspec_debug_branch
    HIPCHK(h, hipStreamSynchronize(h->st));
    std::memcpy(h->pin, ids, 4 * (size_t)n);
    HIPCHK(h, hipMemcpyAsync(s.Y + (size_t)seq * h->d.max_ctx, h->pin, 4 * (size_t)n, hipMemcpyHostToDevice, h->st));
    int r = init_seq(h, seq, n, s.ro_tok);
    if (r) return r;
    int32_t tok = -1;
    HIPCHK(h, hipMemcpyAsync(&tok, s.ro_tok, 4, hipMemcpyDeviceToHost, h->st));
    if ((r = check_err(h))) return r;
    h->prompt_len[seq] = n;
    h->first_tok[seq] = tok;
    if (first_tok) *first_tok = tok;
    return LOOPSPEC_OK;
}

int loopspec_rewind(loopspec_t h, int32_t seq) {
    if (!h) return LOOPSPEC_EINVAL;
    if (seq < 0 || seq >= h->d.max_seqs) return fail(h, LOOPSPEC_EINVAL, "seq out of range");
    if (h->prompt_len[seq] <= 0) return fail(h, LOOPSPEC_ESTATE, "sequence was never prefilled");
    int32_t* tok = (int32_t*)h->pin;
    HIPCHK(h, hipStreamSynchronize(h->st));
    tok[0] = h->first_tok[seq];
    HIPCHK(h, hipMemcpyAsync(h->sch.ro_tok, tok, 4, hipMemcpyHostToDevice, h->st));
    int r = init_seq(h, seq, h->prompt_len[seq], h->sch.ro_tok);
    if (r) return r;
    HIPCHK(h, hipStreamSynchronize(h->st));
    return LOOPSPEC_OK;
}

// Mark the prefilled sequences live with a commit target and rebuild the rows.
static int start_decode(loopspec_t h, int mode, int n_tokens, std::vector<int>& ncommit0) {
    if (!h->bound) return fail(h, LOOPSPEC_ESTATE, "weights are not bound");
    const int Q = h->d.max_seqs;
    Sched& s = h->sch;
    std::vector<int32_t> nc(Q), st(Q, SEQ_EMPTY), tg(Q, 0);
    HIPCHK(h, hipMemcpyAsync(nc.data(), s.q_ncommit, 4 * Q, hipMemcpyDeviceToHost, h->st));
    HIPCHK(h, hipStreamSynchronize(h->st));
    bool any = false;
    for (int q = 0; q < Q; ++q) {
        if (h->prompt_len[q] <= 0) {
            nc[q] = 0;
            continue;
        }
        if (mode != h->tree_mode && !h->fresh[q])
            return fail(h, LOOPSPEC_ESTATE, "decoding mode changed mid-sequence: call loopspec_rewind first");
        if (n_tokens > 0 && h->prompt_len[q] + nc[q] + n_tokens + 2 > h->d.max_ctx)
            return fail(h, LOOPSPEC_ECAPACITY, "sequence would exceed max_ctx");
        st[q] = SEQ_LIVE;
        tg[q] = nc[q] + n_tokens;
        any = true;
    }
    if (!any) return fail(h, LOOPSPEC_ESTATE, "no prefilled sequence");
    ncommit0.assign(nc.begin(), nc.end());
    int32_t zero = 0;
    HIPCHK(h, hipMemcpyAsync(s.q_state, st.data(), 4 * Q, hipMemcpyHostToDevice, h->st));
    HIPCHK(h, hipMemcpyAsync(s.q_target, tg.data(), 4 * Q, hipMemcpyHostToDevice, h->st));
    HIPCHK(h, hipMemcpyAsync(h->mode, &mode, 4, hipMemcpyHostToDevice, h->st));
    HIPCHK(h, hipMemcpyAsync(s.err, &zero, 4, hipMemcpyHostToDevice, h->st));
    hipError_t e = launch_sched(s, OP_REBUILD, 0, 0, nullptr, h->st);
    if (e != hipSuccess) return fail(h, LOOPSPEC_EHIP, hipGetErrorString(e));
    HIPCHK(h, hipStreamSynchronize(h->st));
    h->tree_mode = mode;
    for (int q = 0; q < Q; ++q) {
        if (st[q] != SEQ_LIVE) continue;
        h->fresh[q] = 0;
        for (int r = 1; r <= h->c.R; ++r) {
            const bool ro = r == h->c.R || (mode == MODE_LOOPSPEC && (r == h->c.d1 || (h->c.d2 && r == h->c.d2)));
            if (!ro) h->coda_cov[q][r] = 0;
        }
    }
    return ensure_graph(h);
}

static int run_until(loopspec_t h, int mode, int n_tokens, const std::vector<int>& nc0, int32_t* out) {
    const int Q = h->d.max_seqs;
    Sched& s = h->sch;
    std::vector<int32_t> nc(Q);
    HIPCHK(h, hipEventRecord(h->ev0, h->st));
    long long launched = 0;
    const long long cap = (long long)(n_tokens + 2) * h->c.R * 4 + 64;
    for (;;) {
        HIPCHK(h, hipMemcpyAsync(nc.data(), s.q_ncommit, 4 * Q, hipMemcpyDeviceToHost, h->st));
        HIPCHK(h, hipStreamSynchronize(h->st));
        int remaining = 0;
        for (int q = 0; q < Q; ++q)
            if (h->prompt_len[q] > 0) {
                const int left = nc0[q] + n_tokens - nc[q];
                if (left > 0) remaining = remaining ? std::min(remaining, left) : left;
            }
        if (!remaining) break;
        int r = check_err(h);
        if (r) return r;
        int k = mode == MODE_LOOPSPEC ? std::max(1, (remaining - 1) * h->c.d1) : remaining * h->c.R;
        int i = 0;
        for (; i + kStepsPerGraph <= k && h->exec4; i += kStepsPerGraph) HIPCHK(h, hipGraphLaunch(h->exec4, h->st));
        for (; i < k; ++i) HIPCHK(h, hipGraphLaunch(h->exec, h->st));
        launched += k;
        if (launched > cap) return fail(h, LOOPSPEC_ESTATE, "decode made no progress");
    }
    HIPCHK(h, hipEventRecord(h->ev1, h->st));
    HIPCHK(h, hipEventSynchronize(h->ev1));
    HIPCHK(h, hipEventElapsedTime(&h->last_ms, h->ev0, h->ev1));
    int r = check_err(h);
    if (r) return r;
    if (out) {
        std::vector<int32_t> Y((size_t)Q * h->d.max_ctx);
        HIPCHK(h, hipMemcpy(Y.data(), s.Y, Y.size() * 4, hipMemcpyDeviceToHost));
        for (int q = 0; q < Q; ++q) {
            if (h->prompt_len[q] <= 0) continue;
            // generated token k (1-based count) sits at position prompt_len + k - 1
            const int base = h->prompt_len[q] + nc0[q];
            for (int i = 0; i < n_tokens; ++i) out[(size_t)q * n_tokens + i] = Y[(size_t)q * h->d.max_ctx + base + i];
        }
    }
    return LOOPSPEC_OK;
}

int loopspec_decode(loopspec_t h, int32_t n_tokens, int32_t* out) {
    if (!h) return LOOPSPEC_EINVAL;
    if (n_tokens < 0) return fail(h, LOOPSPEC_EINVAL, "n_tokens < 0");
    std::vector<int> nc0;
    int r = start_decode(h, MODE_LOOPSPEC, n_tokens, nc0);
    if (r) return r;
    return run_until(h, MODE_LOOPSPEC, n_tokens, nc0, out);
}

int loopspec_vanilla_decode(loopspec_t h, int32_t n_tokens, int32_t* out) {
    if (!h) return LOOPSPEC_EINVAL;
    if (n_tokens < 0) return fail(h, LOOPSPEC_EINVAL, "n_tokens < 0");
    std::vector<int> nc0;
    int r = start_decode(h, MODE_VANILLA, n_tokens, nc0);
    if (r) return r;
    return run_until(h, MODE_VANILLA, n_tokens, nc0, out);
}

int loopspec_decode_step(loopspec_t h, int32_t* tok_out, int32_t* src_out) {
    if (!h) return LOOPSPEC_EINVAL;
    const int Q = h->d.max_seqs;
    Sched& s = h->sch;
    // one step with a target far enough away that nothing pauses
    std::vector<int32_t> nc(Q);
    HIPCHK(h, hipMemcpyAsync(nc.data(), s.q_ncommit, 4 * Q, hipMemcpyDeviceToHost, h->st));
    HIPCHK(h, hipStreamSynchronize(h->st));
    std::vector<int> nc0;
    int room = h->d.max_ctx;
    for (int q = 0; q < Q; ++q)
        if (h->prompt_len[q] > 0) room = std::min(room, h->d.max_ctx - h->prompt_len[q] - nc[q] - 2);
    if (room < 1) return fail(h, LOOPSPEC_ECAPACITY, "sequence would exceed max_ctx");
    int r = start_decode(h, MODE_LOOPSPEC, 1, nc0);
    if (r) return r;
    HIPCHK(h, hipGraphLaunch(h->exec, h->st));
    std::vector<int32_t> lt(Q), ls(Q);
    HIPCHK(h, hipMemcpyAsync(lt.data(), s.q_last_tok, 4 * Q, hipMemcpyDeviceToHost, h->st));
    HIPCHK(h, hipMemcpyAsync(ls.data(), s.q_last_src, 4 * Q, hipMemcpyDeviceToHost, h->st));
    if ((r = check_err(h))) return r;
    for (int q = 0; q < Q; ++q) {
        if (tok_out) tok_out[q] = lt[q];
        if (src_out) src_out[q] = ls[q];
    }
    return LOOPSPEC_OK;
}

int loopspec_forced_readout(loopspec_t h, int32_t seq, const int32_t* ids, int32_t n, float* logits_out,
                            int32_t* argmax_out) {
    if (!h) return LOOPSPEC_EINVAL;
    if (seq < 0 || seq >= h->d.max_seqs) return fail(h, LOOPSPEC_EINVAL, "seq out of range");
    if (h->prompt_len[seq] <= 0) return fail(h, LOOPSPEC_ESTATE, "sequence was never prefilled");
    if (!ids || n < 1) return fail(h, LOOPSPEC_EINVAL, "need at least one forced token");
    for (int i = 0; i < n; ++i)
        if (ids[i] < 0 || ids[i] >= h->d.vocab) return fail(h, LOOPSPEC_EINVAL, "token id out of range");
    const int n0 = h->prompt_len[seq], R = h->c.R, V = h->d.vocab, ctx = h->d.max_ctx;
    if (n0 + n + 2 > ctx) return fail(h, LOOPSPEC_ECAPACITY, "forced tokens exceed max_ctx");
    Sched& s = h->sch;
    // the forced continuation, by position: ids[0] at n0, ids[k] at n0 + k
    std::vector<int32_t> f(ctx, 0);
    for (int k = 1; k < n; ++k) f[n0 + k] = ids[k];
    HIPCHK(h, hipMemcpy(s.forced + (size_t)seq * ctx, f.data(), 4 * ctx, hipMemcpyHostToDevice));
    int32_t* tok = (int32_t*)h->pin;
    HIPCHK(h, hipStreamSynchronize(h->st));
    tok[0] = ids[0];
    HIPCHK(h, hipMemcpyAsync(s.ro_tok, tok, 4, hipMemcpyHostToDevice, h->st));
    int r = init_seq(h, seq, n0, s.ro_tok);
    if (r) return r;
    // other sequences stay paused
    const int Q = h->d.max_seqs;
    std::vector<int32_t> st(Q, SEQ_PAUSED), tg(Q, 0);
    for (int q = 0; q < Q; ++q)
        if (h->prompt_len[q] <= 0) st[q] = SEQ_EMPTY;
    st[seq] = SEQ_LIVE;
    tg[seq] = 1 + n;
    const int mode = MODE_FORCED;
    int32_t zero = 0;
    HIPCHK(h, hipMemcpyAsync(s.q_state, st.data(), 4 * Q, hipMemcpyHostToDevice, h->st));
    HIPCHK(h, hipMemcpyAsync(s.q_target, tg.data(), 4 * Q, hipMemcpyHostToDevice, h->st));
    HIPCHK(h, hipMemcpyAsync(h->mode, &mode, 4, hipMemcpyHostToDevice, h->st));
    HIPCHK(h, hipMemcpyAsync(s.err, &zero, 4, hipMemcpyHostToDevice, h->st));
    hipError_t e = launch_sched(s, OP_REBUILD, 0, 0, nullptr, h->st);
    if (e != hipSuccess) return fail(h, LOOPSPEC_EHIP, hipGetErrorString(e));
    h->tree_mode = MODE_FORCED;
    h->fresh[seq] = 0;
    if ((r = ensure_graph(h))) return r;
    for (int k = 0; k < n; ++k)
        for (int d = 1; d <= R; ++d) {
            HIPCHK(h, hipGraphLaunch(h->exec, h->st));
            if (logits_out)
                HIPCHK(h, hipMemcpyAsync(logits_out + ((size_t)k * R + (d - 1)) * V, h->logits, 4 * (size_t)V,
                                         hipMemcpyDeviceToHost, h->st));
            if (argmax_out)
                HIPCHK(h, hipMemcpyAsync(argmax_out + (size_t)k * R + (d - 1), s.ro_tok, 4, hipMemcpyDeviceToHost,
                                         h->st));
            HIPCHK(h, hipStreamSynchronize(h->st));
        }
    return check_err(h);
}

// Whether (d1, d2) can replace the handle's pair now: 0, or the error code
// with its reason in *why.
static int depths_check(loopspec_t h, int d1, int d2, std::string* why) {
    const int R = h->c.R;
    auto no = [&](int code, const std::string& m) {
        *why = m;
        return code;
    };
    if (!h->bound) return no(LOOPSPEC_ESTATE, "weights are not bound");
    if (d1 < 1 || d1 >= R) return no(LOOPSPEC_EINVAL, "need 1 <= d1 < R");
    if (d2 != 0 && !(d1 < d2 && d2 < R)) return no(LOOPSPEC_EINVAL, "need d1 < d2 < R, or d2 = 0");
    if (h->c.second_proposal != LOOPSPEC_SP_GATED && d2 == 0)
        return no(LOOPSPEC_EINVAL, "the ungated second-proposal variants need d2 > 0");
    if (R / d1 >= kChainMax) return no(LOOPSPEC_EINVAL, "R / d1 must be below " + std::to_string(kChainMax));
    const int worst = std::max(worst_case_tree(R, d1, d2, 1), worst_case_tree(R, d1, d2, 2));
    if ((long long)worst * h->d.max_seqs > h->S)
        return no(LOOPSPEC_ECAPACITY, "the pair's worst-case tree (" + std::to_string(worst) + " branches x " +
                                          std::to_string(h->d.max_seqs) + " sequences) exceeds the " +
                                          std::to_string(h->S) + " branch slots");
    if (h->g.Lc)
        for (int q = 0; q < h->d.max_seqs; ++q) {
            if (h->prompt_len[q] <= 0) continue;
            for (int r : {d1, d2})
                if (r > 0 && !h->coda_cov[q][r])
                    return no(LOOPSPEC_ESTATE, "sequence " + std::to_string(q) +
                                                   " has generated positions without coda keys / values at depth " +
                                                   std::to_string(r) + ": switch to it after a prefill or rewind");
        }
    return LOOPSPEC_OK;
}

int loopspec_can_set_depths(loopspec_t h, int32_t d1, int32_t d2) {
    if (!h) return LOOPSPEC_EINVAL;
    std::string why;
    return depths_check(h, d1, d2, &why);
}

int loopspec_set_depths(loopspec_t h, int32_t d1, int32_t d2) {
    if (!h) return LOOPSPEC_EINVAL;
    std::string why;
    if (int r = depths_check(h, d1, d2, &why)) return fail(h, r, why);
    const int R = h->c.R;
    const int worst = std::max(worst_case_tree(R, d1, d2, 1), worst_case_tree(R, d1, d2, 2));
    if (d1 == h->c.d1 && d2 == h->c.d2) return LOOPSPEC_OK;
    h->c.d1 = d1;
    h->c.d2 = d2;
    h->worst = worst;
    Sched& s = h->sch;
    s.d1 = d1;
    s.d2 = d2;
    int32_t zero = 0;
    HIPCHK(h, hipMemcpyAsync(s.err, &zero, 4, hipMemcpyHostToDevice, h->st));
    hipError_t e;
    for (int q = 0; q < h->d.max_seqs; ++q) {
        if (h->prompt_len[q] <= 0) continue;
        if ((e = launch_sched(s, OP_RESET, q, 0, nullptr, h->st)) != hipSuccess ||
            (e = launch_embed(h->g, s.js, s.njs, 1, h->embed, h->bf16, h->X, h->st)) != hipSuccess ||
            (h->g.Lp && (e = enqueue_stack(h, STACK_PRE, s.rowsP, s.nP, h->S, false)) != hipSuccess))
            return fail(h, LOOPSPEC_EHIP, hipGetErrorString(e));
    }
    drop_graphs(h);
    return check_err(h);
}

int loopspec_vanilla_step(loopspec_t h, int32_t* tok_out) {
    if (!h) return LOOPSPEC_EINVAL;
    std::vector<int> nc0;
    int r = start_decode(h, MODE_VANILLA, 1, nc0);
    if (r) return r;
    const int Q = h->d.max_seqs;
    std::vector<int32_t> out(Q, -1);
    if ((r = run_until(h, MODE_VANILLA, 1, nc0, out.data()))) return r;
    if (tok_out)
        for (int q = 0; q < Q; ++q) tok_out[q] = h->prompt_len[q] > 0 ? out[q] : -1;
    return LOOPSPEC_OK;
}

}  // extern "C"

namespace {

// Host copy of the branch tables (between calls only).
struct HostTree {
    std::vector<int32_t> active, seq, pos, tok, depth, parent, x1, x2, gate, tdone;
};

int read_tree(loopspec_t h, HostTree& t) {
    const Sched& s = h->sch;
    const int S = h->S;
    std::vector<int32_t>* v[] = {&t.active, &t.seq, &t.pos, &t.tok, &t.depth, &t.parent, &t.x1, &t.x2, &t.gate};
    const int32_t* src[] = {s.s_active, s.s_seq, s.s_pos, s.s_tok, s.s_depth, s.s_parent, s.s_x1, s.s_x2, s.s_gate};
    for (int i = 0; i < 9; ++i) {
        v[i]->assign(S, 0);
        HIPCHK(h, hipMemcpyAsync(v[i]->data(), src[i], 4 * (size_t)S, hipMemcpyDeviceToHost, h->st));
    }
    t.tdone.assign(h->d.max_seqs, 0);
    HIPCHK(h, hipMemcpyAsync(t.tdone.data(), s.q_tdone, 4 * (size_t)h->d.max_seqs, hipMemcpyDeviceToHost, h->st));
    HIPCHK(h, hipStreamSynchronize(h->st));
    return LOOPSPEC_OK;
}

// Row of branch `slot` at `depth` reading from X row `xrow`, with its chain of
// in-flight ancestors (positions tdone .. pos-1).
int branch_row(loopspec_t h, const HostTree& t, int slot, int depth, int xrow, Row* out) {
    Row r{};
    r.xrow = xrow;
    r.slot = slot;
    r.seq = t.seq[slot];
    r.pos = t.pos[slot];
    r.depth = depth;
    r.tdone = t.tdone[r.seq];
    r.src = xrow;
    int x = t.parent[slot];
    for (int p = r.pos - 1; p >= r.tdone; --p) {
        if (p - r.tdone >= kChainMax || x < 0 || x >= h->S)
            return fail(h, LOOPSPEC_ESTATE, "inconsistent branch tree");
        r.anc[p - r.tdone] = x;
        x = t.parent[x];
    }
    *out = r;
    return LOOPSPEC_OK;
}

}  // namespace

extern "C" {

int loopspec_debug_branch(loopspec_t h, int32_t slot, loopspec_branch* info, int32_t* prefix) {
    if (!h || !info) return LOOPSPEC_EINVAL;
    if (slot < 0 || slot >= h->S) return fail(h, LOOPSPEC_EINVAL, "slot out of range");
    HostTree t;
    int r = read_tree(h, t);
    if (r) return r;
    loopspec_branch b{};
    b.active = t.active[slot] ? 1 : 0;
    b.seq = b.pos = b.depth = b.token = b.parent = b.tdone = b.x1 = b.x2 = -1;
    b.gate = 0;
    if (b.active) {
        b.seq = t.seq[slot];
        b.pos = t.pos[slot];
        b.depth = t.depth[slot];
        b.token = t.tok[slot];
        b.parent = t.parent[slot];
        b.tdone = t.tdone[b.seq];
        b.x1 = t.x1[slot];
        b.x2 = t.x2[slot];
        b.gate = t.gate[slot];
    }
    *info = b;
    if (!b.active || !prefix) return LOOPSPEC_OK;
    // positions < tdone: the sequence's token record (prompt, committed tokens)
    if (b.tdone > 0) {
        HIPCHK(h, hipMemcpyAsync(prefix, h->sch.Y + (size_t)b.seq * h->d.max_ctx, 4 * (size_t)b.tdone,
                                 hipMemcpyDeviceToHost, h->st));
        HIPCHK(h, hipStreamSynchronize(h->st));
    }
    // positions tdone .. pos: the branch and its in-flight ancestors, up to the root
    int x = slot;
    for (int p = b.pos; p >= b.tdone; --p) {
        if (x < 0 || x >= h->S) return fail(h, LOOPSPEC_ESTATE, "inconsistent branch tree");
        prefix[p] = t.tok[x];
        x = t.parent[x];
    }
    if (x != -1) return fail(h, LOOPSPEC_ESTATE, "inconsistent branch tree");
    return LOOPSPEC_OK;
}

int loopspec_debug_readout(loopspec_t h, int32_t slot, int32_t depth, float* logits) {
    if (!h || !logits) return LOOPSPEC_EINVAL;
    if (!h->bound) return fail(h, LOOPSPEC_ESTATE, "weights are not bound");
    if (slot < 0 || slot >= h->S) return fail(h, LOOPSPEC_EINVAL, "slot out of range");
    HostTree t;
    int r = read_tree(h, t);
    if (r) return r;
    if (!t.active[slot]) return fail(h, LOOPSPEC_ESTATE, "slot holds no branch");
    const int cur = t.depth[slot];
    if (depth < 1 || depth > cur)
        return fail(h, LOOPSPEC_EINVAL, "depth must lie in 1.." + std::to_string(cur) + ", the branch's current depth");
    if (h->g.Lc) {
        // coda caches of in-flight positions exist at the readout depths of the
        // tree's schedule only
        const int m = h->tree_mode;
        const bool ok = m == MODE_FORCED || depth == h->c.R ||
                        (m == MODE_LOOPSPEC && (depth == h->c.d1 || (h->c.d2 && depth == h->c.d2)));
        if (!ok) return fail(h, LOOPSPEC_EINVAL, "a model with coda blocks reads out only at its readout depths");
    }
    const int R = h->c.R, xr = h->xrow_pf;
    // staged rows: [0..R] the branch at depth 0..R, [R+1] the readout row
    std::vector<Row> rows(R + 2);
    for (int d = 0; d <= R; ++d)
        if ((r = branch_row(h, t, slot, d, xr, &rows[d]))) return r;
    rows[R + 1] = rows[depth];
    if (depth == cur) rows[R + 1].src = slot;             // the branch's own state, copied
    HIPCHK(h, hipStreamSynchronize(h->st));
    Row* rp = (Row*)h->pin;
    std::memcpy(rp, rows.data(), sizeof(Row) * rows.size());
    int32_t* misc = (int32_t*)(rp + rows.size());
    misc[0] = 1;
    misc[1] = 1;
    misc[2] = xr;
    misc[3] = t.tok[slot];
    HIPCHK(h, hipMemcpyAsync(h->pf_rows, rp, sizeof(Row) * rows.size(), hipMemcpyHostToDevice, h->st));
    HIPCHK(h, hipMemcpyAsync(h->pf_n, misc, 8, hipMemcpyHostToDevice, h->st));
    HIPCHK(h, hipMemcpyAsync(h->pf_jobs, misc + 2, 8, hipMemcpyHostToDevice, h->st));
    const Row* rd = h->pf_rows;
    const int32_t* one = h->pf_n;
    hipError_t e = hipSuccess;
    if (depth == cur) {
        e = launch_copy_rows(h->g, rd + R + 1, one, 1, h->X, h->st);
    } else {
        // recompute the branch's newest token from its embedding up to `depth`
        // through the same launches a decode step uses (batch-invariant kernels:
        // the keys and values it rewrites are the ones already there)
        e = launch_embed(h->g, h->pf_jobs, one, 1, h->embed, h->bf16, h->X, h->st);
        if (e == hipSuccess && h->g.Lp) e = enqueue_stack(h, STACK_PRE, rd, one, h->S, false);
        for (int d = 1; d <= depth && e == hipSuccess; ++d) e = enqueue_stack(h, STACK_CORE, rd + d, one, h->S, false);
    }
    if (e == hipSuccess && h->g.Lc) e = enqueue_stack(h, STACK_CODA, rd + R + 1, one, h->S, false);
    if (e == hipSuccess) e = enqueue_head(h, rd + R + 1, one, h->S);
    if (e != hipSuccess) return fail(h, LOOPSPEC_EHIP, hipGetErrorString(e));
    HIPCHK(h, hipMemcpyAsync(logits, h->logits, 4 * (size_t)h->d.vocab, hipMemcpyDeviceToHost, h->st));
    return check_err(h);
}

int loopspec_decode_profile(loopspec_t h, int32_t n_tokens, int32_t kind, int32_t max_launches, float* ms_out,
                            int32_t* info_out, int32_t* n_out) {
    if (!h || !n_out || n_tokens < 0 || max_launches < 0 || (max_launches && (!ms_out || !info_out)))
        return LOOPSPEC_EINVAL;
    if (kind < LOOPSPEC_PROF_PASS || kind > LOOPSPEC_PROF_HEAD) return fail(h, LOOPSPEC_EINVAL, "unknown kernel kind");
    if (kind == LOOPSPEC_PROF_PASS && !h->pass_on)
        return fail(h, LOOPSPEC_EINVAL, "decode passes of this handle run as per-kernel launches");
    if (kind != LOOPSPEC_PROF_PASS && kind != LOOPSPEC_PROF_HEAD && h->pass_on)
        return fail(h, LOOPSPEC_EINVAL, "decode passes of this handle run as the persistent pass kernel");
    std::vector<int> nc0;
    int r = start_decode(h, MODE_LOOPSPEC, n_tokens, nc0);
    if (r) return r;
    const int Q = h->d.max_seqs, S = h->S;
    const int per_step = std::max(2, 2 * std::max(h->g.Lb, 1));
    while ((int)h->prof_ev.size() < per_step) {
        hipEvent_t e = nullptr;
        HIPCHK(h, hipEventCreate(&e));
        h->prof_ev.push_back(e);
    }
    Sched& s = h->sch;
    std::vector<int32_t> nc(Q);
    std::vector<Row> rows(S);
    int32_t nrow[2] = {0, 0};
    int count = 0, step = 0;
    const long long cap = (long long)(n_tokens + 2) * h->c.R * 4 + 64;
    for (;;) {
        HIPCHK(h, hipMemcpyAsync(nc.data(), s.q_ncommit, 4 * Q, hipMemcpyDeviceToHost, h->st));
        HIPCHK(h, hipMemcpyAsync(nrow, s.nB, 8, hipMemcpyDeviceToHost, h->st));
        HIPCHK(h, hipMemcpyAsync(rows.data(), s.rowsB, sizeof(Row) * S, hipMemcpyDeviceToHost, h->st));
        HIPCHK(h, hipStreamSynchronize(h->st));
        bool left = false;
        for (int q = 0; q < Q; ++q)
            if (h->prompt_len[q] > 0 && nc[q] < nc0[q] + n_tokens) left = true;
        if (!left) break;
        if (++step > cap) return fail(h, LOOPSPEC_ESTATE, "decode made no progress");
        // this step's pass: rows, and the key/value positions it must read --
        // committed positions once per (sequence, depth), in-flight positions
        // once per (slot holding the position, depth)
        const int M = std::min(nrow[0], S);
        long long kvpos = 0;
        std::vector<std::pair<int, int>> seen_c, seen_s;
        for (int i = 0; i < M; ++i) {
            const Row& x = rows[i];
            const std::pair<int, int> c{x.seq, x.depth};
            if (std::find(seen_c.begin(), seen_c.end(), c) == seen_c.end()) {
                seen_c.push_back(c);
                kvpos += x.tdone;
            }
            for (int p = x.tdone; p <= x.pos; ++p) {
                const int slot = p == x.pos ? x.slot : x.anc[p - x.tdone];
                const std::pair<int, int> a{slot, x.depth};
                if (std::find(seen_s.begin(), seen_s.end(), a) == seen_s.end()) {
                    seen_s.push_back(a);
                    kvpos += 1;
                }
            }
        }
        h->prof_kind = kind;
        h->prof_n = 0;
        hipError_t e = enqueue_step(h);
        h->prof_kind = -1;
        if (e != hipSuccess) return fail(h, LOOPSPEC_EHIP, hipGetErrorString(e));
        HIPCHK(h, hipStreamSynchronize(h->st));
        for (int i = 0; i + 1 < h->prof_n; i += 2) {
            if (count < max_launches) {
                float ms = 0.f;
                HIPCHK(h, hipEventElapsedTime(&ms, h->prof_ev[i], h->prof_ev[i + 1]));
                ms_out[count] = ms;
                info_out[3 * count] = kind == LOOPSPEC_PROF_HEAD ? nrow[1] : M;
                info_out[3 * count + 1] = kind == LOOPSPEC_PROF_HEAD ? 0 : (int32_t)kvpos;
                info_out[3 * count + 2] = step - 1;
            }
            ++count;
        }
        if ((r = check_err(h))) return r;
    }
    *n_out = count;
    return LOOPSPEC_OK;
}

int loopspec_time_kernels(loopspec_t h, int32_t M, int32_t reps, float* ms_out) {
    if (!h || !ms_out) return LOOPSPEC_EINVAL;
    if (M < 1 || M > h->S || reps < 1) return fail(h, LOOPSPEC_EINVAL, "need 1 <= M <= slots and reps >= 1");
    if (!h->bound || h->prompt_len[0] <= 0) return fail(h, LOOPSPEC_ESTATE, "prefill sequence 0 first");
    const int pos = h->prompt_len[0];
    // M branch rows at the sequence's current length, spread over the depths
    std::vector<Row> rows(M);
    for (int i = 0; i < M; ++i) {
        Row r{};
        r.xrow = i;
        r.slot = i;
        r.seq = 0;
        r.pos = pos;
        r.depth = 1 + i % h->c.R;
        r.tdone = pos;
        r.src = i;
        rows[i] = r;
    }
    HIPCHK(h, hipStreamSynchronize(h->st));
    std::memcpy(h->pin, rows.data(), sizeof(Row) * M);
    ((int32_t*)(h->pin + sizeof(Row) * 64))[0] = M;
    HIPCHK(h, hipMemcpyAsync(h->pf_rows, h->pin, sizeof(Row) * M, hipMemcpyHostToDevice, h->st));
    HIPCHK(h, hipMemcpyAsync(h->pf_n, h->pin + sizeof(Row) * 64, 4, hipMemcpyHostToDevice, h->st));
    const int L = h->g.Lb;
    std::vector<hipEvent_t> ev((size_t)reps * L * 5 + 1);
    for (auto& e : ev) HIPCHK(h, hipEventCreate(&e));
    size_t n = 0;
    {
        hipError_t e = launch_gather(h->g, h->pf_rows, h->pf_n, M, h->X, h->pb, h->bf16, h->st);
        if (e != hipSuccess) return fail(h, LOOPSPEC_EHIP, hipGetErrorString(e));
    }
    HIPCHK(h, hipEventRecord(ev[n++], h->st));
    for (int r = 0; r < reps; ++r)
        for (int l = 0; l < L; ++l)
            for (int k = 0; k < 5; ++k) {
                hipError_t e = enqueue_kernel(h, k, STACK_CORE, l, h->pf_rows, h->pf_n, h->S, false);
                if (e != hipSuccess) return fail(h, LOOPSPEC_EHIP, hipGetErrorString(e));
                HIPCHK(h, hipEventRecord(ev[n++], h->st));
            }
    HIPCHK(h, hipStreamSynchronize(h->st));
    double acc[5] = {0, 0, 0, 0, 0};
    for (size_t i = 1; i < n; ++i) {
        float ms = 0.f;
        HIPCHK(h, hipEventElapsedTime(&ms, ev[i - 1], ev[i]));
        acc[(i - 1) % 5] += ms;
    }
    for (auto& e : ev) (void)hipEventDestroy(e);
    for (int k = 0; k < 5; ++k) ms_out[k] = (float)(acc[k] / ((double)reps * L));
    return check_err(h);
}

int loopspec_time_pass(loopspec_t h, int32_t M, int32_t reps, float* ms_out, int32_t* fused_out) {
    if (!h || !ms_out) return LOOPSPEC_EINVAL;
    if (M < 1 || M > h->S || reps < 1) return fail(h, LOOPSPEC_EINVAL, "need 1 <= M <= slots and reps >= 1");
    if (!h->bound || h->prompt_len[0] <= 0) return fail(h, LOOPSPEC_ESTATE, "prefill sequence 0 first");
    const int pos = h->prompt_len[0];
    std::vector<Row> rows(M);
    for (int i = 0; i < M; ++i) {
        Row r{};
        r.xrow = i;
        r.slot = i;
        r.seq = 0;
        r.pos = pos;
        r.depth = 1 + i % h->c.R;
        r.tdone = pos;
        r.src = i;
        rows[i] = r;
    }
    HIPCHK(h, hipStreamSynchronize(h->st));
    std::memcpy(h->pin, rows.data(), sizeof(Row) * M);
    ((int32_t*)(h->pin + sizeof(Row) * 64))[0] = M;
    HIPCHK(h, hipMemcpyAsync(h->pf_rows, h->pin, sizeof(Row) * M, hipMemcpyHostToDevice, h->st));
    HIPCHK(h, hipMemcpyAsync(h->pf_n, h->pin + sizeof(Row) * 64, 4, hipMemcpyHostToDevice, h->st));
    // as in a decode step: the preparation kernel (pass) or the gather kernel
    // (per-kernel path) in front of every pass, outside the timing
    const bool fused = h->pass_on;
    const PassParams pp = pass_params(h, STACK_CORE, h->pf_rows, h->pf_n);
    std::vector<hipEvent_t> ev((size_t)2 * reps);
    for (auto& e : ev) HIPCHK(h, hipEventCreate(&e));
    for (int r = 0; r < reps; ++r) {
        hipError_t e = fused ? launch_pass_prep(pp, h->bf16, M, h->st)
                             : launch_gather(h->g, h->pf_rows, h->pf_n, M, h->X, h->pb, h->bf16, h->st);
        if (e != hipSuccess) return fail(h, LOOPSPEC_EHIP, hipGetErrorString(e));
        HIPCHK(h, hipEventRecord(ev[2 * r], h->st));
        if (fused) {
            e = launch_pass(pp, h->bf16, h->pass_grid, h->st);
        } else {
            for (int l = 0; l < h->g.Lb && e == hipSuccess; ++l)
                for (int k = 0; k < 5 && e == hipSuccess; ++k)
                    e = enqueue_kernel(h, k, STACK_CORE, l, h->pf_rows, h->pf_n, h->S, false);
        }
        if (e != hipSuccess) return fail(h, LOOPSPEC_EHIP, hipGetErrorString(e));
        HIPCHK(h, hipEventRecord(ev[2 * r + 1], h->st));
    }
    HIPCHK(h, hipStreamSynchronize(h->st));
    double acc = 0.0;
    for (int r = 0; r < reps; ++r) {
        float ms = 0.f;
        HIPCHK(h, hipEventElapsedTime(&ms, ev[2 * r], ev[2 * r + 1]));
        acc += ms;
    }
    for (auto& e : ev) (void)hipEventDestroy(e);
    *ms_out = (float)(acc / reps);
    if (fused_out) *fused_out = fused ? 1 : 0;
    return check_err(h);
}

int loopspec_set_seed(loopspec_t h, uint64_t seed) {
    if (!h) return LOOPSPEC_EINVAL;
    HIPCHK(h, hipStreamSynchronize(h->st));
    HIPCHK(h, hipMemcpy((void*)h->sch.seed, &seed, 8, hipMemcpyHostToDevice));
    h->c.seed = seed;
    return LOOPSPEC_OK;
}

int loopspec_get_stats(loopspec_t h, loopspec_stats* out) {
    if (!h || !out) return LOOPSPEC_EINVAL;
    long long v[ST_N];
    HIPCHK(h, hipMemcpyAsync(v, h->sch.stats, sizeof(v), hipMemcpyDeviceToHost, h->st));
    HIPCHK(h, hipStreamSynchronize(h->st));
    out->steps = v[ST_STEPS];
    out->committed = v[ST_COMMITTED];
    out->n_acc1 = v[ST_ACC1];
    out->n_acc2 = v[ST_ACC2];
    out->n_restart = v[ST_RESTART];
    out->gate_eval = v[ST_GATE_EVAL];
    out->gate_open = v[ST_GATE_OPEN];
    out->sum_M = v[ST_SUM_M];
    out->max_M = v[ST_MAX_M];
    out->spawn_refused = v[ST_REFUSED];
    out->zero_mass = v[ST_ZERO_MASS];
    out->tv_d1 = v[ST_TV1];
    out->tv_d2 = v[ST_TV2];
    out->tv_count = v[ST_TVN];
    for (int i = 0; i < 65; ++i) out->hist_M[i] = v[ST_HIST + i];
    return LOOPSPEC_OK;
}

int loopspec_reset_stats(loopspec_t h) {
    if (!h) return LOOPSPEC_EINVAL;
    HIPCHK(h, hipMemsetAsync(h->sch.stats, 0, ST_N * 8, h->st));
    HIPCHK(h, hipStreamSynchronize(h->st));
    return LOOPSPEC_OK;
}

int loopspec_last_decode_ms(loopspec_t h, float* ms) {
    if (!h || !ms) return LOOPSPEC_EINVAL;
    *ms = h->last_ms;
    return LOOPSPEC_OK;
}

int loopspec_pass_kernel(loopspec_t h, int32_t* on) {
    if (!h || !on) return LOOPSPEC_EINVAL;
    *on = !h->pass_on ? 0 : h->chunks_cap <= kPassAttnWgChunks ? 1 : 2;
    return LOOPSPEC_OK;
}

int loopspec_capacity(loopspec_t h, int32_t* slots, int32_t* worst) {
    if (!h) return LOOPSPEC_EINVAL;
    if (slots) *slots = h->S;
    if (worst) *worst = h->worst;
    return LOOPSPEC_OK;
}

}  // extern "C"
