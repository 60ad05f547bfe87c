// Device-resident LoopSpec scheduler and the kernels that feed it.
//
// The scheduler carries out the bookkeeping of Alg. 1 between two batched
// recurrent passes, entirely on the GPU so a whole decode step can be replayed
// as one graph with no host round trip:
//   * every branch of the pass advanced one depth;
//   * the root that reached R commits the token chosen by Verify (readout
//     kernels decided it) and the set is re-rooted at the chosen child
//     (Reroot: keep c* and its descendants, free the rest); its KV for every
//     depth moves to the committed cache at its position;
//   * a branch that reached d1 spawns a child on X || x1; a branch that reached
//     d2 with an open gate spawns a second child on X || x2 (Spawn);
//   * the row lists of the next pass are rebuilt: every live branch (B rows),
//     the branches whose next depth is a readout depth (C rows), and the
//     freshly spawned branches (P rows, for prelude blocks).
// Verification and re-rooting are applied before the proposals of the same
// step; a child spawned this step inside a pruned subtree would be dropped in
// the same step, so skipping it gives the same branch set (Alg. 1 order).
#include "ls_sched.h"

#include <algorithm>

namespace ls {

// ---------------------------------------------------------------------------
// scheduler (single thread: the tree holds at most 64 branches)
// ---------------------------------------------------------------------------
__device__ static int alloc_slot(const Sched& s) {
    for (int i = 0; i < s.g.S; ++i)
        if (!s.s_active[i]) return i;
    return -1;
}

__device__ static void init_slot(const Sched& s, int c, int q, int pos, int tok, int parent) {
    s.s_active[c] = 1;
    s.s_seq[c] = q;
    s.s_pos[c] = pos;
    s.s_tok[c] = tok;
    s.s_depth[c] = 0;
    s.s_parent[c] = parent;
    s.s_c1[c] = -1;
    s.s_c2[c] = -1;
    s.s_x1[c] = -1;
    s.s_x2[c] = -1;
    s.s_gate[c] = 0;
}

__device__ static bool in_subtree(const Sched& s, int x, int c) {
    if (c < 0) return false;
    for (int k = 0; x >= 0 && k <= s.g.S; ++k) {
        if (x == c) return true;
        x = s.s_parent[x];
    }
    return false;
}

__device__ static void fill_chain(const Sched& s, int slot, int tdone, Row& r) {
    int x = s.s_parent[slot];
    for (int p = s.s_pos[slot] - 1; p >= tdone; --p) {
        if (p - tdone >= kChainMax || x < 0) {         // inconsistent tree: never index out of range
            atomicOr(s.err, ERR_SLOTS);
            break;
        }
        r.anc[p - tdone] = x;
        x = s.s_parent[x];
    }
}

__device__ static bool is_readout(const Sched& s, int mode, int d) {
    if (mode == MODE_FORCED) return d >= 1 && d <= s.R;
    if (mode == MODE_VANILLA) return d == s.R;
    return d == s.d1 || (s.d2 > 0 && d == s.d2) || d == s.R;
}

__global__ void k_sched(Sched s, int op, int op_seq, int op_pos, const int32_t* op_tok) {
    if (threadIdx.x != 0) return;
    const int mode = *s.mode;
    const int S = s.g.S, ctx = s.g.max_ctx;
    long long* st = s.stats;
    int njc = 0, njs = 0;

    if (op == OP_STEP) {
        const int nB = *s.nB, nC = *s.nC;
        for (int i = 0; i < nB; ++i) s.s_depth[s.rowsB[i].slot] += 1;
        if (nB > 0) {
            st[ST_STEPS] += 1;
            st[ST_SUM_M] += nB;
            if (nB > st[ST_MAX_M]) st[ST_MAX_M] = nB;
            st[ST_HIST + (nB < 64 ? nB : 64)] += 1;
        }
        for (int q = 0; q < s.max_seqs; ++q) {
            s.q_last_tok[q] = -1;
            s.q_last_src[q] = -1;
        }
        // ---- gate statistics: Alg. 1 evaluates the gate of every branch that
        //      reaches d2 this step, before the root's verification prunes any
        if (mode == MODE_LOOPSPEC && s.d2 > 0) {
            for (int i = 0; i < nC; ++i) {
                if (s.rowsC[i].depth != s.d2) continue;
                st[ST_GATE_EVAL] += 1;
                st[ST_GATE_OPEN] += s.ro_aux[i] ? 1 : 0;
            }
        }
        // ---- roots at depth R: commit, re-root, prune -----------------------
        for (int i = 0; i < nC; ++i) {
            const Row row = s.rowsC[i];
            if (row.depth != s.R) continue;
            const int q = row.seq, b = row.slot, np = row.pos + 1;
            int tok = s.ro_tok[i], src = s.ro_aux[i];
            if (mode == MODE_FORCED) {
                tok = s.forced[(size_t)q * ctx + np];
                src = 0;
            } else if (mode == MODE_VANILLA) {
                src = 0;
            }
            s.Y[(size_t)q * ctx + np] = tok;
            s.q_ncommit[q] += 1;
            s.q_last_tok[q] = tok;
            s.q_last_src[q] = src;
            st[ST_COMMITTED] += 1;
            if (mode == MODE_LOOPSPEC) st[src == 1 ? ST_ACC1 : src == 2 ? ST_ACC2 : ST_RESTART] += 1;
            // greedy: TV between one-hot readouts is the argmax mismatch (the
            // argmax at d2 is kept in s_x2 whether or not its branch was
            // spawned; the sampled readout adds its TV sums itself)
            if (mode == MODE_LOOPSPEC && s.greedy && s.s_x1[b] >= 0) {
                const int x1 = s.s_x1[b], a2 = s.s_x2[b] >= 0 ? s.s_x2[b] : x1;
                st[ST_TVN] += 1;
                st[ST_TV1] += x1 != tok ? (1LL << 32) : 0;
                if (s.d2 > 0) st[ST_TV2] += a2 != tok ? (1LL << 32) : 0;
            }
            int c = src == 1 ? s.s_c1[b] : src == 2 ? s.s_c2[b] : -1;
            s.jc[3 * njc] = q;
            s.jc[3 * njc + 1] = b;
            s.jc[3 * njc + 2] = row.pos;
            ++njc;
            for (int x = 0; x < S; ++x)
                if (s.s_active[x] && s.s_seq[x] == q && !in_subtree(s, x, c)) s.s_active[x] = 0;
            s.q_tdone[q] = np;
            if (np >= ctx - 1) {                       // no room for another position
                atomicOr(s.err, ERR_CTX);
                s.q_state[q] = SEQ_PAUSED;
                for (int x = 0; x < S; ++x)
                    if (s.s_seq[x] == q) s.s_active[x] = 0;
                s.q_root[q] = -1;
                continue;
            }
            if (c < 0) {
                c = alloc_slot(s);
                if (c < 0) {                           // cannot happen: the old root was just freed
                    atomicOr(s.err, ERR_SLOTS);
                    s.q_state[q] = SEQ_PAUSED;
                    s.q_root[q] = -1;
                    continue;
                }
                init_slot(s, c, q, np, tok, -1);
                s.js[2 * njs] = c;
                s.js[2 * njs + 1] = tok;
                ++njs;
            }
            s.s_parent[c] = -1;
            s.q_root[q] = c;
            if (s.q_ncommit[q] >= s.q_target[q]) s.q_state[q] = SEQ_PAUSED;
        }
        // ---- proposals at d1 / d2 -----------------------------------------------
        if (mode == MODE_LOOPSPEC) {
            for (int i = 0; i < nC; ++i) {
                const Row row = s.rowsC[i];
                const int b = row.slot, q = row.seq;
                // the branch must still hold this slot: a slot pruned above may
                // already carry a new root (depth 0) of the same step.  A
                // sequence that reached its commit target in this step still
                // records its drafts (it resumes from this tree on the next
                // call); one whose tree was dropped has no active slot left.
                if (!s.s_active[b] || s.s_seq[b] != q || s.s_pos[b] != row.pos || s.s_depth[b] != row.depth ||
                    s.q_root[q] < 0)
                    continue;
                if (row.depth == s.d1) {
                    const int x1 = s.ro_tok[i];
                    s.s_x1[b] = x1;
                    s.s_c2[b] = -1;
                    s.s_gate[b] = 0;
                    const int c = row.pos + 1 < ctx - 1 ? alloc_slot(s) : -1;
                    s.s_c1[b] = c;
                    if (c < 0) {
                        st[ST_REFUSED] += 1;
                        continue;
                    }
                    init_slot(s, c, q, row.pos + 1, x1, b);
                    s.js[2 * njs] = c;
                    s.js[2 * njs + 1] = x1;
                    ++njs;
                } else if (s.d2 > 0 && row.depth == s.d2) {
                    if (s.greedy) s.s_x2[b] = s.ro_tok[i];   // verification reads it only with the gate open
                    if (!s.ro_aux[i]) continue;
                    const int x2 = s.ro_tok[i];
                    const int c = row.pos + 1 < ctx - 1 ? alloc_slot(s) : -1;
                    if (c < 0) {                       // no room: the gate stays closed
                        st[ST_REFUSED] += 1;
                        continue;
                    }
                    s.s_gate[b] = 1;
                    s.s_x2[b] = x2;
                    s.s_c2[b] = c;
                    init_slot(s, c, q, row.pos + 1, x2, b);
                    s.js[2 * njs] = c;
                    s.js[2 * njs + 1] = x2;
                    ++njs;
                }
            }
        }
    } else if (op == OP_RESET) {
        // new proposal depths: drop every speculative branch of the sequence
        // and its root's drafts.  A root below the new d1 keeps the depths it
        // has computed (they do not depend on d1, d2); one at or past it
        // restarts at depth 0 from its embedding, so that it drafts at the new
        // d1 (its hidden states and slot keys / values are recomputed)
        const int q = op_seq, c = s.q_root[q];
        if (c >= 0) {
            for (int x = 0; x < S; ++x)
                if (x != c && s.s_active[x] && s.s_seq[x] == q) s.s_active[x] = 0;
            const int depth = s.s_depth[c];
            init_slot(s, c, q, s.s_pos[c], s.s_tok[c], -1);
            if (depth < s.d1) {
                s.s_depth[c] = depth;
            } else {
                s.js[0] = c;
                s.js[1] = s.s_tok[c];
                njs = 1;
            }
        }
    } else if (op == OP_INIT) {
        const int q = op_seq, n = op_pos, tok = op_tok[0];
        for (int x = 0; x < S; ++x)
            if (s.s_seq[x] == q) s.s_active[x] = 0;
        const int c = alloc_slot(s);
        if (c < 0) {
            atomicOr(s.err, ERR_SLOTS);
        } else {
            init_slot(s, c, q, n, tok, -1);
            s.q_root[q] = c;
            s.q_tdone[q] = n;
            s.q_ncommit[q] = 1;
            s.q_state[q] = SEQ_PAUSED;
            s.Y[(size_t)q * ctx + n] = tok;
            s.js[0] = c;
            s.js[1] = tok;
            njs = 1;
        }
    }

    // ---- next pass: rows of every live branch, grouped by sequence -------------
    int nB = 0, nC = 0, nP = 0;
    for (int q = 0; q < s.max_seqs; ++q) {
        if (s.q_state[q] != SEQ_LIVE) continue;
        const int tdone = s.q_tdone[q];
        for (int x = 0; x < S; ++x) {
            if (!s.s_active[x] || s.s_seq[x] != q) continue;
            Row r;
            r.xrow = x;
            r.slot = x;
            r.seq = q;
            r.pos = s.s_pos[x];
            r.depth = s.s_depth[x] + 1;
            r.tdone = tdone;
            r.src = x;                                   // copy source for readout rows
            r.pad = 0;
            fill_chain(s, x, tdone, r);
            s.rowsB[nB++] = r;
            if (is_readout(s, mode, r.depth)) {
                if (s.coda_xrow0 >= 0) r.xrow = s.coda_xrow0 + nC;
                s.rowsC[nC++] = r;
            }
        }
    }
    for (int j = 0; j < njs; ++j) {
        const int x = s.js[2 * j];
        const int q = s.s_seq[x];
        Row r;
        r.xrow = x;
        r.slot = x;
        r.seq = q;
        r.pos = s.s_pos[x];
        r.depth = 0;
        r.tdone = s.q_tdone[q];
        r.src = x;
        r.pad = 0;
        fill_chain(s, x, r.tdone, r);
        s.rowsP[nP++] = r;
    }
    *s.nB = nB;
    *s.nC = nC;
    *s.nP = nP;
    *s.njc = njc;
    *s.njs = njs;
}

hipError_t launch_sched(const Sched& s, int op, int op_seq, int op_pos, const int32_t* op_tok, hipStream_t st) {
    hipLaunchKernelGGL(k_sched, dim3(1), dim3(64), 0, st, s, op, op_seq, op_pos, op_tok);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// greedy readout: arg-max over the per-tile maxima, then the step's decision
// for the row (draft at d1, gate + second proposal at d2, cascade at R)
// ---------------------------------------------------------------------------
__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
    return v > bv || (v == bv && i < bi) || bi < 0;
}

__global__ void __launch_bounds__(256) k_finalize_greedy(Sched s, int fin_op, const float* tmax,
                                                          const int32_t* targ, int tiles) {
    const int i = blockIdx.x;
    if (i >= *s.nC) return;
    __shared__ float sv[256];
    __shared__ int si[256];
    float bv = -INFINITY;
    int bi = -1;
    for (int t = threadIdx.x; t < tiles; t += 256) {
        const float v = tmax[(size_t)i * tiles + t];
        const int id = targ[(size_t)i * tiles + t];
        if (better(v, id, bv, bi)) {
            bv = v;
            bi = id;
        }
    }
    sv[threadIdx.x] = bv;
    si[threadIdx.x] = bi;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if (threadIdx.x < o) {
            const float v = sv[threadIdx.x + o];
            const int id = si[threadIdx.x + o];
            if (id >= 0 && better(v, id, sv[threadIdx.x], si[threadIdx.x])) {
                sv[threadIdx.x] = v;
                si[threadIdx.x] = id;
            }
        }
        __syncthreads();
    }
    if (threadIdx.x != 0) return;
    const int a = si[0];
    const Row row = s.rowsC[i];
    const int mode = *s.mode;
    int aux = 0;
    if (fin_op == FIN_STEP && mode == MODE_LOOPSPEC) {
        const int b = row.slot;
        if (row.depth == s.d2 && s.d2 > 0) {
            aux = a != s.s_x1[b];                               // greedy gate: argmax q2~ != x1
        } else if (row.depth == s.R) {
            aux = a == s.s_x1[b] ? 1 : (s.s_gate[b] && a == s.s_x2[b]) ? 2 : 0;
        }
    }
    s.ro_tok[i] = a;
    s.ro_aux[i] = aux;
}

// ---------------------------------------------------------------------------
// P for Ouro-style models: H^(0) = E[x]
// ---------------------------------------------------------------------------
template <typename WT>
__device__ __forceinline__ void embed_job(const Geo& g, const int32_t* jobs, int j, const WT* E, float* X) {
    const int xrow = jobs[2 * j], tok = jobs[2 * j + 1];
    const WT* e = E + (size_t)tok * g.h;
    float* x = X + (size_t)xrow * g.h;
    for (int k = threadIdx.x; k < g.h; k += blockDim.x)
        x[k] = sizeof(WT) == 2 ? bf2f(((const uint16_t*)e)[k]) : ((const float*)e)[k];
}

template <typename WT>
__global__ void __launch_bounds__(256) k_embed(Geo g, const int32_t* jobs, const int32_t* njobs, const WT* E,
                                               float* X) {
    const int j = blockIdx.x;
    if (j >= *njobs) return;
    embed_job<WT>(g, jobs, j, E, X);
}

hipError_t launch_embed(const Geo& g, const int32_t* jobs, const int32_t* njobs, int jobs_cap, const void* E,
                        bool bf16, float* X, hipStream_t st) {
    if (bf16)
        hipLaunchKernelGGL(k_embed<uint16_t>, dim3(jobs_cap), dim3(256), 0, st, g, jobs, njobs,
                           (const uint16_t*)E, X);
    else
        hipLaunchKernelGGL(k_embed<float>, dim3(jobs_cap), dim3(256), 0, st, g, jobs, njobs, (const float*)E, X);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// pass buffers: the rounded hidden state and its RMSNorm statistics, in the
// row order of the pass (the partials are the ones the residual epilogue writes)
// ---------------------------------------------------------------------------
template <typename WT>
__global__ void __launch_bounds__(256) k_gather(Geo g, const Row* rows, const int32_t* nrows, const float* X,
                                                PassBuf pb) {
    const int m = blockIdx.x;
    if (m >= *nrows) return;
    const float* x = X + (size_t)rows[m].xrow * g.h;
    for (int t = threadIdx.x; t < g.ssq_tiles; t += blockDim.x) {
        float v[16];
#pragma unroll
        for (int c = 0; c < 16; ++c) v[c] = x[t * 16 + c];
        pb.SSQR[(size_t)m * g.ssq_tiles + t] = ssq16(v);
#pragma unroll
        for (int c = 0; c < 16; ++c) {
            if (sizeof(WT) == 2)
                ((uint16_t*)pb.XB)[(size_t)m * g.h + t * 16 + c] = f2h(v[c]);
            else
                ((float*)pb.XB)[(size_t)m * g.h + t * 16 + c] = v[c];
        }
    }
}

hipError_t launch_gather(const Geo& g, const Row* rows, const int32_t* nrows, int rows_cap, const float* X,
                         PassBuf pb, bool bf16, hipStream_t st) {
    if (bf16)
        hipLaunchKernelGGL(k_gather<uint16_t>, dim3(rows_cap), dim3(128), 0, st, g, rows, nrows, X, pb);
    else
        hipLaunchKernelGGL(k_gather<float>, dim3(rows_cap), dim3(128), 0, st, g, rows, nrows, X, pb);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// KV commit: the verified root's keys/values of every depth move to the
// committed cache at its position (they are needed by every later position)
// ---------------------------------------------------------------------------
// commit job j, table t (of g.T), keys (kv = 0) or values (kv = 1)
__device__ __forceinline__ void commit_job(const Sched& s, int j, int t, int kv, char* kvc, const char* kvs,
                                           int wbytes) {
    const int q = s.jc[3 * j], b = s.jc[3 * j + 1], pos = s.jc[3 * j + 2];
    const u32x4* src = (const u32x4*)(kvs + kvs_index(s.g, b, t, kv) * wbytes);
    const int per_head = s.g.dh * wbytes / 16;        // 16-byte vectors per head slice
    const int n = s.g.H * per_head;
    for (int k = threadIdx.x; k < n; k += blockDim.x) {
        const int head = k / per_head, i = k - head * per_head;
        u32x4* dst = (u32x4*)(kvc + kvc_index(s.g, q, t, kv, head, pos) * wbytes);
        dst[i] = src[k];
    }
}

__global__ void __launch_bounds__(256) k_kv_commit(Sched s, char* kvc, const char* kvs, int wbytes) {
    const int j = blockIdx.y;
    if (j >= *s.njc) return;
    commit_job(s, j, blockIdx.x >> 1, blockIdx.x & 1, kvc, kvs, wbytes);
}

hipError_t launch_kv_commit(const Sched& s, void* kvc, const void* kvs, int wbytes, hipStream_t st) {
    hipLaunchKernelGGL(k_kv_commit, dim3(s.g.T * 2, s.max_seqs), dim3(256), 0, st, s, (char*)kvc,
                       (const char*)kvs, wbytes);
    return hipGetLastError();
}

// The two independent tails of a decode step in one launch: rows y <
// max_seqs of the grid copy the committed roots' keys and values (as
// k_kv_commit), row y = max_seqs embeds the spawned branches' tokens (as
// k_embed); x covers max(2 T, slots).
template <typename WT>
__global__ void __launch_bounds__(256) k_commit_embed(Sched s, char* kvc, const char* kvs, int wbytes, const WT* E,
                                                      float* X) {
    const int y = blockIdx.y, x = blockIdx.x;
    if (y < s.max_seqs) {
        if (y < *s.njc && x < 2 * s.g.T) commit_job(s, y, x >> 1, x & 1, kvc, kvs, wbytes);
    } else if (x < *s.njs) {
        embed_job<WT>(s.g, s.js, x, E, X);
    }
}

hipError_t launch_commit_embed(const Sched& s, void* kvc, const void* kvs, int wbytes, const void* E, bool bf16,
                               float* X, hipStream_t st) {
    const dim3 grid(std::max(2 * s.g.T, s.g.S), s.max_seqs + 1);
    if (bf16)
        hipLaunchKernelGGL(k_commit_embed<uint16_t>, grid, dim3(256), 0, st, s, (char*)kvc, (const char*)kvs, wbytes,
                           (const uint16_t*)E, X);
    else
        hipLaunchKernelGGL(k_commit_embed<float>, grid, dim3(256), 0, st, s, (char*)kvc, (const char*)kvs, wbytes,
                           (const float*)E, X);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// readout copies for coda blocks: X[row.xrow] = X[row.src]; the coda transforms
// a copy so the branch's own hidden state keeps recurring
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256) k_copy_rows(Geo g, const Row* rows, const int32_t* nrows, float* X) {
    const int i = blockIdx.x;
    if (i >= *nrows) return;
    const int dst = rows[i].xrow, src = rows[i].src;
    for (int k = threadIdx.x; k < g.h; k += blockDim.x) X[(size_t)dst * g.h + k] = X[(size_t)src * g.h + k];
}

hipError_t launch_copy_rows(const Geo& g, const Row* rows, const int32_t* nrows, int rows_cap, float* X,
                            hipStream_t st) {
    hipLaunchKernelGGL(k_copy_rows, dim3(rows_cap), dim3(256), 0, st, g, rows, nrows, X);
    return hipGetLastError();
}

hipError_t launch_finalize_greedy(const Sched& s, int fin_op, const float* tmax, const int32_t* targ, int tiles,
                                  int rows_cap, hipStream_t st) {
    hipLaunchKernelGGL(k_finalize_greedy, dim3(rows_cap), dim3(256), 0, st, s, fin_op, tmax, targ, tiles);
    return hipGetLastError();
}

}  // namespace ls
