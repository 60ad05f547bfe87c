// Device-resident branch scheduler and the small kernels around it
// (ls_sched.hip, ls_sample.hip).
#pragma once
#include "ls_common.h"

namespace ls {

// largest vocabulary the sampling readout holds (ids per thread x threads per row)
constexpr int kSampleMaxVocab = 65536;

enum Mode { MODE_LOOPSPEC = 0, MODE_VANILLA = 1, MODE_FORCED = 2 };
enum SeqState { SEQ_EMPTY = 0, SEQ_LIVE = 1, SEQ_PAUSED = 2 };
// OP_RESET: drop a sequence's speculative branches and restart its root at depth 0
enum SchedOp { OP_STEP = 0, OP_INIT = 1, OP_REBUILD = 2, OP_RESET = 3 };
enum FinOp { FIN_STEP = 0, FIN_TARGET = 1 };

// statistics block (int64)
enum Stat {
    ST_STEPS = 0, ST_COMMITTED, ST_ACC1, ST_ACC2, ST_RESTART, ST_GATE_EVAL, ST_GATE_OPEN,
    ST_SUM_M, ST_MAX_M, ST_REFUSED, ST_ZERO_MASS,
    // TV(p_R, p_d1) and TV(p_R, p_d2) summed over verifications (units of 2^-32), and their count
    ST_TV1, ST_TV2, ST_TVN,
    ST_HIST, ST_N = ST_HIST + 65
};

// error bits
// ERR_TREE: a branch reached a decision its tree does not support (no first draft recorded)
enum ErrBit { ERR_NUMERIC = 1, ERR_CTX = 2, ERR_SLOTS = 4, ERR_SYNC = kErrPoll, ERR_TREE = 16 };

struct Sched {
    Geo g;
    int max_seqs;
    int R, d1, d2;
    int variant;         // second proposal: 0 gated residual, 1 ungated residual, 2 ungated naive (both masked)
    int greedy;
    float temperature, top_p;
    const unsigned long long* seed;   // device: key word 0 of every draw
    const int32_t* mode;
    // branch slots [S]
    int32_t *s_active, *s_seq, *s_pos, *s_tok, *s_depth, *s_parent, *s_c1, *s_c2, *s_x1, *s_x2, *s_gate;
    // sequences [max_seqs]
    int32_t *q_root, *q_tdone, *q_ncommit, *q_target, *q_state, *q_last_tok, *q_last_src;
    int32_t* Y;          // [max_seqs][max_ctx] token at each position
    int32_t* forced;     // [max_seqs][max_ctx] teacher-forced tokens
    // row lists: B (recurrent pass), C (readout rows), P (spawned rows, prelude)
    Row* rowsB; int32_t* nB;
    Row* rowsC; int32_t* nC;
    Row* rowsP; int32_t* nP;
    int coda_xrow0;      // first X row used for readout copies (Raven coda); -1: read X[slot]
    // readout results per C row
    int32_t *ro_tok, *ro_aux;
    // jobs produced by a step
    int32_t *jc, *njc;   // KV commits: (seq, slot, pos)
    int32_t *js, *njs;   // embeddings: (xrow, token)
    long long* stats;
    int32_t* err;
    // sampling state (temperature > 0): per slot proposal distributions
    float *q1, *q2;      // [S][V]
    float* q2t;          // [S][V] the readout distribution at d2 (for TV(p_R, p_d2))
    unsigned long long* srow;   // [S][kRowWords] barrier state of each readout row's shards (ls_sample.h)
};

hipError_t launch_sched(const Sched& s, int op, int op_seq, int op_pos, const int32_t* op_tok,
                        hipStream_t st);
hipError_t launch_finalize(const Sched& s, int fin_op, const float* logits, const float* tmax,
                           const int32_t* targ, int tiles, int rows_cap, hipStream_t st);
hipError_t launch_embed(const Geo& g, const int32_t* jobs, const int32_t* njobs, int jobs_cap,
                        const void* embed, bool bf16, float* X, hipStream_t st);
hipError_t launch_kv_commit(const Sched& s, void* kvc, const void* kvs, int wbytes, hipStream_t st);
// launch_kv_commit and launch_embed of a decode step (the Sched's js / njs jobs) in one launch
hipError_t launch_commit_embed(const Sched& s, void* kvc, const void* kvs, int wbytes, const void* E, bool bf16,
                               float* X, hipStream_t st);
// X[row.xrow] = X[row.src] for every row (readout copies that coda blocks transform)
hipError_t launch_copy_rows(const Geo& g, const Row* rows, const int32_t* nrows, int rows_cap, float* X,
                            hipStream_t st);
// pass buffers of a row list: XB[m] = round(X[xrow]), SSQR[m] = per-tile sums of squares
hipError_t launch_gather(const Geo& g, const Row* rows, const int32_t* nrows, int rows_cap, const float* X,
                         PassBuf pb, bool bf16, hipStream_t st);

}  // namespace ls
