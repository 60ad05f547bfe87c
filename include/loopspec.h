/*
 * loopspec.h — C ABI of the MI355X (gfx950) LoopSpec decode library.
 *
 * LoopSpec: pipelined self-speculative decoding for Looped Transformers.
 * A looped model computes H^(0) = P(X), H^(r) = B(H^(r-1)) for r = 1..R and
 * reads out p_r = C(H^(r)) at any depth (Sec. 3.1, Eq. loop-recurrence).
 * LoopSpec keeps a tree of branches, each a prefix whose newest token sits at
 * its own recurrent depth; every decode step advances all branches by one
 * depth in one batched pass over the shared weights, drafts at depth d1,
 * proposes a gated residual second candidate at d2, and verifies the root at
 * R with cascade rejection sampling (Sec. 4, Alg. 1).  Decoding is lossless
 * under greedy decoding and sampling.
 *
 * Conventions for every call
 *  - Return value: LOOPSPEC_OK (0) or a negative LOOPSPEC_E* code.  On error
 *    loopspec_last_error(h) returns a message owned by the handle, valid until
 *    the next call on that handle.  No exception crosses this boundary.
 *  - Pointers named *_host are host memory owned by the caller; they are read
 *    or written before the call returns.  Device pointers (the weights) are
 *    borrowed: they must stay valid and unmodified for the handle's life.
 *  - All GPU work runs on the stream given to loopspec_create (a hipStream_t
 *    passed as void*).  NULL makes the handle create and own a non-blocking
 *    stream (a decode step is replayed as a captured graph, which the legacy
 *    default stream cannot hold).  Calls that return host results synchronise
 *    that stream before returning.
 *  - A handle is not thread-safe; one host thread at a time.
 *  - Matrices are row-major [out][in] (a row is one output feature).  Weights
 *    are bf16 or fp32 as given by loopspec_dims.weight_dtype.  Token ids are
 *    int32 in [0, vocab).  Positions are 0-based; the prompt of a sequence
 *    occupies positions 0..n-1.
 */
#ifndef LOOPSPEC_H
#define LOOPSPEC_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LOOPSPEC_OK 0
#define LOOPSPEC_EINVAL (-1)    /* bad argument or configuration */
#define LOOPSPEC_ENOMEM (-2)    /* device or host allocation failed */
#define LOOPSPEC_EHIP (-3)      /* a HIP runtime call failed */
#define LOOPSPEC_ECAPACITY (-4) /* context, token or slot capacity exceeded */
#define LOOPSPEC_ESTATE (-5)    /* call not valid in the handle's state */
#define LOOPSPEC_ENUMERIC (-6)  /* NaN/Inf met in the readout logits */

#define LOOPSPEC_F32 0
#define LOOPSPEC_BF16 1

typedef struct loopspec_handle* loopspec_t;

/* Model shape.  P = embedding + n_prelude blocks, B = n_core blocks applied R
 * times, C = n_coda blocks + final RMSNorm + LM head (Sec. 3.1, Fig. 2:
 * Ouro-style models have n_prelude = n_coda = 0).  Blocks are pre-RMSNorm
 * multi-head attention with rotate-half RoPE and a SwiGLU FFN. */
typedef struct {
    int32_t hidden;       /* h = n_heads * head_dim */
    int32_t n_heads;
    int32_t head_dim;     /* 16, 32, 64, 96 or 128 */
    int32_t ffn;          /* SwiGLU width F */
    int32_t vocab;        /* V */
    int32_t n_prelude;
    int32_t n_core;
    int32_t n_coda;
    int32_t weight_dtype; /* LOOPSPEC_F32 or LOOPSPEC_BF16 */
    int32_t tied_head;    /* 1: the LM head is the embedding matrix */
    float rope_base;
    float rms_eps;
    int32_t max_seqs;     /* independent sequences decoded together */
    int32_t max_ctx;      /* positions per sequence (prompt + generated) */
} loopspec_dims;

/* Decoding configuration: total depth R and proposal depths d1 < d2 < R
 * (Alg. 1 input).  d2 = 0 selects the single-proposal pipeline (Sec. 4.2).
 * temperature = 0 selects greedy decoding; otherwise the readout applies
 * temperature then top-p (Sec. 3.1).  seed keys the Philox4x64-10 draws. */
typedef struct {
    int32_t R;
    int32_t d1;
    int32_t d2;
    float temperature;
    float top_p;          /* in (0, 1]; 1 disables the filter */
    uint64_t seed;
    int32_t max_slots;    /* branch slots; 0 = worst case of the tree (all gates open) */
    int32_t per_kernel;   /* 0: a decode pass of a block stack over at most 16 rows runs
                             as one persistent kernel when the model fits it;
                             1: one launch per kernel (QKV, attention, O, gate/up, down) */
    int32_t second_proposal; /* the second-proposal variants of the ablation (Ablation Study,
                             Table 3); sampling only (temperature > 0, d2 > 0):
                             LOOPSPEC_SP_GATED    gated residual proposal q2 = q2~ (-) q1
                                                  (Sec. 4.3; the method, and the default);
                             LOOPSPEC_SP_RESIDUAL ungated: always propose from q2~ (-) q1
                                                  with the first proposal masked out and
                                                  the rest renormalised;
                             LOOPSPEC_SP_NAIVE    ungated: always propose from q2~ with the
                                                  first proposal masked out and renormalised.
                             A masked distribution with no mass left makes no proposal. */
    int32_t shared_prefix;   /* 1: decode attention launched per kernel (per_kernel = 1, or
                             more than 16 slots) runs as shared-prefix tasks: the rows of
                             one sequence at one depth read each committed chunk of keys
                             and values once (KV cache management of the pipelined decode),
                             the work spread over the whole GPU as one-wave tasks whose
                             partials are combined by the task that completes a (row, head);
                             0: one workgroup per (head, row).  Within a handle a row's
                             result does not depend on the rows it is grouped with. */
} loopspec_config;

enum { LOOPSPEC_SP_GATED = 0, LOOPSPEC_SP_RESIDUAL = 1, LOOPSPEC_SP_NAIVE = 2 };

/* Per-block weights (device pointers). */
typedef struct {
    const void* attn_norm; /* [h] */
    const void* wq;        /* [h][h] */
    const void* wk;        /* [h][h] */
    const void* wv;        /* [h][h] */
    const void* wo;        /* [h][h] */
    const void* ffn_norm;  /* [h] */
    const void* wg;        /* [F][h] */
    const void* wu;        /* [F][h] */
    const void* wd;        /* [h][F] */
} loopspec_layer_weights;

typedef struct {
    const void* embed;       /* [V][h] */
    const void* final_norm;  /* [h] */
    const void* head;        /* [V][h]; ignored when tied_head */
    const loopspec_layer_weights* layers; /* host array: prelude, core, coda blocks in order */
    int32_t n_layers;        /* n_prelude + n_core + n_coda */
} loopspec_weights;

/* Statistics since the last loopspec_reset_stats (summed over sequences):
 * commit sources and gate rates (App. on gating and on commitment sources),
 * effective batch per step (number of branches advanced by one B pass). */
typedef struct {
    int64_t steps;          /* B passes launched with at least one branch */
    int64_t committed;      /* tokens committed by Verify (or per vanilla step) */
    int64_t n_acc1;         /* first proposals accepted */
    int64_t n_acc2;         /* second proposals accepted */
    int64_t n_restart;      /* neither accepted: resampled, fresh branch */
    int64_t gate_eval;      /* branches that reached d2 */
    int64_t gate_open;      /* ... whose gate opened (second child spawned) */
    int64_t sum_M;          /* sum over steps of the effective batch */
    int64_t max_M;
    int64_t spawn_refused;  /* proposals that found no free slot */
    int64_t zero_mass;      /* residuals with no positive mass (should stay 0) */
    int64_t tv_d1;          /* sum over verifications of TV(p_R, p_d1) of the verified root,
                               in units of 2^-32 (greedy: 2^32 per argmax mismatch) */
    int64_t tv_d2;          /* the same for TV(p_R, p_d2) (0 without a second proposal) */
    int64_t tv_count;       /* verifications counted in tv_d1 / tv_d2 */
    int64_t hist_M[65];     /* effective batch histogram, last bin = 64+ */
} loopspec_stats;

/* Create a decoder.  Validates the shape (hidden = n_heads*head_dim,
 * head_dim in {16, 32, 64, 96, 128}, hidden and ffn multiples of 32), the depths
 * (1 <= d1 < d2 < R, or d2 = 0 and 1 <= d1 < R; Alg. 1 input) and sizes the
 * branch-slot pool: max_slots = 0 takes the largest tree Alg. 1 can grow when
 * every gate opens (branch-growth recurrence, Sec. 4.3), per sequence.
 * Allocates every device buffer (KV caches per recurrent depth, implementation
 * details) up front; nothing is allocated while decoding.
 * stream: hipStream_t (may be NULL).  Errors: EINVAL, ENOMEM, EHIP,
 * ECAPACITY (more than 64 slots).  On error *out still receives the handle
 * when one was made, so that loopspec_last_error can explain the failure;
 * the caller then destroys it. */
int loopspec_create(const loopspec_dims* dims, const loopspec_config* cfg, void* stream,
                    loopspec_t* out);

/* Bind the model weights (borrowed device pointers, see the struct).  Must
 * precede prefill.  Errors: EINVAL (NULL pointer or wrong layer count). */
int loopspec_bind_weights(loopspec_t h, const loopspec_weights* w);

/* Prefill sequence `seq` with a prompt (Alg. 1 prologue): H <- P(x_{1:n}),
 * R applications of B writing every depth's KV, x ~ C(H) at depth R; the
 * token is committed and a root branch is spawned on x_{1:n} || x at depth 0.
 * ids_host: n token ids; first_tok_host: receives x.  Replaces any previous
 * state of that sequence.  Errors: EINVAL, ECAPACITY (n + 2 > max_ctx: the prompt,
 * the first token and one position of lookahead),
 * ESTATE (weights unbound), ENUMERIC, EHIP. */
int loopspec_prefill(loopspec_t h, int32_t seq, const int32_t* ids_host, int32_t n,
                     int32_t* first_tok_host);

/* Restore sequence `seq` to its state right after its prefill (the committed
 * prompt KV is kept; the branch tree and generated tokens are dropped).
 * Errors: ESTATE if the sequence was never prefilled. */
int loopspec_rewind(loopspec_t h, int32_t seq);

/* One LoopSpec step (Alg. 1 loop body) for every live sequence: all active
 * branches advance one depth in one batched pass; branches at d1 / d2 draft;
 * each root at R verifies and commits one token.  tok_out_host[s] receives
 * the token committed for sequence s this step or -1; n_acc_out_host[s]
 * receives its source (1 first proposal, 2 second, 0 restart) or -1.  Either
 * pointer may be NULL.  Errors: ESTATE, ECAPACITY (context full), EHIP. */
int loopspec_decode_step(loopspec_t h, int32_t* tok_out_host, int32_t* n_acc_out_host);

/* Decode until every prefilled sequence has committed n_tokens more tokens,
 * replaying the captured one-step hipGraph.  out_host: [max_seqs][n_tokens]
 * (row s holds sequence s's new tokens; rows of sequences not prefilled are
 * left untouched).  n_tokens = 0 does nothing.  Errors: EINVAL (n_tokens < 0),
 * ESTATE, ECAPACITY (prompt length + tokens committed so far, the prefill's
 * included, + n_tokens + 2 would exceed max_ctx for some sequence; checked
 * before any launch, the sequences are then left as they were), EHIP, ENUMERIC. */
int loopspec_decode(loopspec_t h, int32_t n_tokens, int32_t* out_host);

/* Vanilla looped decoding on the same kernels (Fig. 1a): all R depths of one
 * token, then its readout at R, then the next token.  Same contract as
 * loopspec_decode; greedy results are bit-identical to it. */
int loopspec_vanilla_decode(loopspec_t h, int32_t n_tokens, int32_t* out_host);

/* Teacher-forced readouts on the vanilla schedule: after a prefill of `seq`,
 * appends the n tokens ids_host one position at a time (all R depths each),
 * recording the readout logits C(H^(r)) at every depth r = 1..R for the
 * prefix ending at each appended token.  logits_host: [n][R][V] fp32 or NULL;
 * argmax_host: [n][R] or NULL.  The sequence's branch tree is dropped
 * (call loopspec_rewind to decode again).  Errors: EINVAL, ECAPACITY,
 * ESTATE, EHIP. */
int loopspec_forced_readout(loopspec_t h, int32_t seq, const int32_t* ids_host, int32_t n,
                            float* logits_host, int32_t* argmax_host);

/* One vanilla token for every prefilled sequence (Fig. 1a, on the same
 * kernels and graphs as loopspec_vanilla_decode): R recurrent steps, the
 * readout at depth R and its draw.  tok_out_host[s] receives sequence s's
 * token, -1 for sequences never prefilled (may be NULL).  The first call after
 * a prefill or rewind fixes the sequence to the vanilla schedule; greedy
 * tokens are bit-identical to loopspec_decode's.  Errors: ESTATE (no prefilled
 * sequence, or a sequence mid-way through LoopSpec decoding), ECAPACITY, EHIP,
 * ENUMERIC. */
int loopspec_vanilla_step(loopspec_t h, int32_t* tok_out_host);

/* Switch the proposal depths (d1, d2) of Alg. 1 between decode calls, for a
 * planner that re-fits the power-law TV envelope (Sec. 4.1, Observation) from
 * the tv_d1 / tv_d2 statistics and minimises Theorem 2's bound while decoding.
 * Same rules as at creation (1 <= d1 < d2 < R, or d2 = 0; the ungated
 * variants need d2 > 0; R / d1 below the chain limit), and the pair's
 * worst-case tree times max_seqs must fit the branch-slot pool sized at
 * creation.  Every prefilled sequence drops its speculative branches and its
 * root's drafts; a root that has not reached the new d1 keeps its computed
 * depths, one at or past it restarts at depth 0 (its hidden states are
 * recomputed from its embedding).  Committed tokens and caches are kept, so
 * decoding stays lossless across the switch; the step graphs are captured
 * again by the next decode call.  The same pair again does nothing.
 * Models with coda blocks: a readout at depth r runs the coda over the
 * prefix's coda keys / values at depth r, which a decode writes only at its
 * own readout depths (d1, d2, R) for the positions it commits; once a
 * sequence has generated positions, a new d1 or d2 must be a depth that
 * every decode of it so far has read out at (after a prefill or rewind any
 * pair is allowed: the prompt holds every depth).
 * Errors: EINVAL, ECAPACITY, ESTATE (weights unbound, or coda keys / values
 * missing at a new depth), EHIP. */
int loopspec_set_depths(loopspec_t h, int32_t d1, int32_t d2);

/* What loopspec_set_depths(h, d1, d2) would return right now, without
 * changing anything (0: the switch is allowed); for planners choosing among
 * pairs.  Does not set the last-error text. */
int loopspec_can_set_depths(loopspec_t h, int32_t d1, int32_t d2);

/* A branch of the decoding tree (Alg. 1: a prefix whose newest token sits at
 * its own recurrent depth). */
typedef struct {
    int32_t active;   /* 1 when the slot holds a live branch; the other fields are -1 (gate 0) if not */
    int32_t seq;      /* its sequence */
    int32_t pos;      /* position of its newest token */
    int32_t depth;    /* recurrent depth that token has reached (0 right after a spawn) */
    int32_t token;    /* the newest token */
    int32_t parent;   /* parent branch's slot, -1 for the root */
    int32_t tdone;    /* committed length of the sequence: positions < tdone are committed;
                         the root sits at position tdone */
    int32_t x1, x2;   /* the drafts it recorded at d1 and d2 (-1: none yet) */
    int32_t gate;     /* 1 when its gate opened at d2 (a second child was spawned) */
} loopspec_branch;

/* Inspect branch slot `slot` between calls.  prefix_host (may be NULL):
 * receives the branch's whole token prefix, positions 0..pos (the prompt, the
 * committed tokens, then the in-flight ancestors from the root down to the
 * branch itself), i.e. pos + 1 ids.  Errors: EINVAL (slot outside the pool),
 * ESTATE (inconsistent tree), EHIP. */
int loopspec_debug_branch(loopspec_t h, int32_t slot, loopspec_branch* info_host, int32_t* prefix_host);

/* Readout logits C(H^(depth)) of the newest token of the branch in `slot`,
 * for any depth 1..its current depth (Alg. 1: q1 = C(H^(d1)) at the first
 * proposal, q2~ = C(H^(d2)) at the gate, p_R at verification; Sec. 3.1,
 * Eq. loop-recurrence).  At the current depth the branch's own hidden state
 * is read out; below it the token is recomputed from its embedding through
 * the same launches a decode step uses (the kernels are batch-invariant, so
 * the keys and values it rewrites are bit-identical to those present).
 * Models with coda blocks read out only at depths whose coda caches exist for
 * in-flight positions: d1, d2 and R under LoopSpec decoding, R under vanilla.
 * logits_host: [vocab] fp32.  Call between decode calls.  Errors: EINVAL (slot,
 * depth), ESTATE (empty slot, weights unbound), EHIP, ENUMERIC. */
int loopspec_debug_readout(loopspec_t h, int32_t slot, int32_t depth, float* logits_host);

/* Replace the Philox key word `seed` used by every later draw (sampling
 * only; greedy decoding draws nothing).  Already-committed tokens are kept;
 * call loopspec_rewind to resample a continuation.  Errors: EHIP. */
int loopspec_set_seed(loopspec_t h, uint64_t seed);

/* Copy the statistics out / zero them. */
int loopspec_get_stats(loopspec_t h, loopspec_stats* out_host);
int loopspec_reset_stats(loopspec_t h);

/* Time (ms, HIP events on the handle's stream) of the last decode or
 * vanilla_decode call, from its first step launch to its last step's end. */
int loopspec_last_decode_ms(loopspec_t h, float* ms_out_host);

/* Measurement: average duration in ms of one launch of each kernel of the
 * batched recurrent pass, timed with HIP events on the handle's stream around
 * each launch of `reps` full passes over the core blocks with M branch rows
 * (1 <= M <= slots) at sequence 0's current context length.
 * ms_out_host[5]: RMSNorm+QKV(+RoPE, KV write), attention (+combine),
 * O projection (+residual), RMSNorm+gate/up(+SwiGLU), down (+residual).
 * Overwrites branch hidden states and slot KV: call loopspec_rewind before
 * decoding again.  Errors: EINVAL, ESTATE (no prefilled sequence 0), EHIP. */
int loopspec_time_kernels(loopspec_t h, int32_t M, int32_t reps, float* ms_out_host);

/* Kernel kinds of loopspec_decode_profile. */
enum {
    LOOPSPEC_PROF_PASS = 0,   /* the persistent decode pass of the core block stack (one launch per step) */
    LOOPSPEC_PROF_QKV = 1,    /* per-kernel path, core blocks: RMSNorm + QKV + RoPE + KV write */
    LOOPSPEC_PROF_ATTN = 2,   /* attention */
    LOOPSPEC_PROF_O = 3,      /* O projection + residual */
    LOOPSPEC_PROF_GU = 4,     /* RMSNorm + gate/up + SwiGLU */
    LOOPSPEC_PROF_DOWN = 5,   /* down projection + residual */
    LOOPSPEC_PROF_HEAD = 6    /* final RMSNorm + LM head of the readout rows */
};

/* Measurement aid: decode like loopspec_decode (same kernels, same launch
 * configurations, same tokens), but with every step's kernels launched
 * directly instead of replaying the step graph, and each launch of kernel
 * `kind` carrying a pair of HIP events in its own dispatch
 * (hipExtLaunchKernel), which take the kernel's start and end times, as a
 * kernel trace does (LOOPSPEC_PROF_*; the
 * pass kinds must match how this handle runs its decode passes, see
 * loopspec_pass_kernel).  For launch i < max_launches: ms_host[i] its
 * duration; info_host[3i..3i+2] = (rows M of the launch, key/value positions
 * the step's rows read -- each committed position once per (sequence, depth),
 * each in-flight position once per (branch slot, depth); 0 for the LM head --,
 * the decode step it belongs to).  *n_out receives the number of launches
 * (which may exceed max_launches).  Errors: as loopspec_decode, EINVAL for a
 * kind this handle does not launch. */
int loopspec_decode_profile(loopspec_t h, int32_t n_tokens, int32_t kind, int32_t max_launches, float* ms_host,
                            int32_t* info_host, int32_t* n_out);

/* Mean duration (ms, HIP events on the handle's stream) of one launch of the
 * decode pass of the shared (core) block stack over M synthetic branch rows at
 * the length of prefilled sequence 0, in the launch configuration decoding
 * uses (the persistent pass kernel when enabled, else the per-kernel
 * launches of every block).  *fused_out = 1 when the persistent kernel ran.
 * Same side effects and errors as loopspec_time_kernels. */
int loopspec_time_pass(loopspec_t h, int32_t M, int32_t reps, float* ms_out_host, int32_t* fused_out_host);

/* Slots in the branch pool and the worst-case effective batch per sequence
 * for (R, d1, d2); sizes checked by the tests. */
int loopspec_capacity(loopspec_t h, int32_t* slots_host, int32_t* worst_per_seq_host);

/* *on = 0 when decode passes of this handle run as per-kernel launches,
 * else the persistent pass kernel runs them (per_kernel = 0, at most 16
 * slots, and the model's kinds fit one work item per CU) and *on tells its
 * attention: 1 = one workgroup per (row, head), for contexts of at most
 * 32 chunks of 64 positions (max_ctx <= 2048); 2 = (row, head, chunk) tasks
 * over every CU, combined through device memory, for longer contexts. */
int loopspec_pass_kernel(loopspec_t h, int32_t* on_host);

const char* loopspec_last_error(loopspec_t h);

/* Free every buffer, graph and event of the handle.  NULL is ignored. */
void loopspec_destroy(loopspec_t h);

/* Largest effective batch (active branches of one sequence) Alg. 1 can reach
 * for (R, d1, d2) when every gate opens and every verification accepts a
 * proposal; for d1 | d2 and d1 | R it equals the branch-growth bound
 * B = sum_{k < R/d1} s_k with s_k = s_{k-1} + s_{k-d2/d1} (Sec. 4.3; 249 at
 * (32, 2, 8)).  Host-only, no GPU call.  Returns -1 for invalid depths and
 * for pairs the library does not run (R / d1 of 24 or more: a branch would
 * carry more in-flight ancestors than a pass row holds). */
int32_t loopspec_worst_case_branches(int32_t R, int32_t d1, int32_t d2);

/* Measurement aid beside the method: the HBM read rate of a plain stream,
 * the practical ceiling for the weight stream of a decode pass.  Reads the
 * caller's device buffer buf_dev[0 .. bytes) reps + 1 times (the first pass
 * untimed) with 16-byte nontemporal loads from 256 workgroups of 256
 * threads, on `stream` (a hipStream_t, may be NULL), and waits for it.
 * xor_out_dev: caller-owned device memory of 65536 uint32; thread t writes
 * the XOR of the 32-bit words it read in the last pass, so the XOR of all
 * 65536 equals the XOR of the whole buffer.  *gbps_host = bytes * reps /
 * elapsed, in GB/s.  bytes: a positive multiple of 16 below 2^36.  Needs no
 * handle and allocates nothing on the device.  Errors: EINVAL, EHIP. */
int loopspec_read_bandwidth(const void* buf_dev, uint64_t bytes, int32_t reps, void* stream,
                            uint32_t* xor_out_dev, float* gbps_host);

/* ---------------------------------------------------------------------------
 * Standalone proposal / verification decisions (Alg. 1: Spawn at d1 and d2,
 * Verify at R; Sec. 4.2-4.3) for independent keyed positions, on the same
 * vocabulary-sharded sampling kernels a decode step runs.  Row i stands for a
 * branch whose readout logits at d1, d2 and R are z1, z2, zR (row i of each at
 * offset i * z_stride floats; z_stride 0 gives every row the same logits).
 * For every row, with distributions after temperature then top-p (Sec. 3.1):
 *   q1 = dist(z1), x1 ~ q1 (Philox event DRAFT1);
 *   q2~ = dist(z2); the second proposal per cfg.second_proposal (gated:
 *   only when q2~(x1) < q1(x1), from q2 = q2~ (-) q1, Eq. adaptive-gate and
 *   Eq. residual-proposal; the ablation's ungated variants as in
 *   loopspec_config), x2 ~ q2 (event DRAFT2);
 *   p = dist(zR); cascade verification: accept x1 iff U1 < min(1, p/q1 at
 *   x1) (event ACC1); else rho = p (-) q1 and, with a second proposal, accept
 *   x2 iff U2 < min(1, rho/q2 at x2) (event ACC2); else x ~ rho (-) q2, or
 *   x ~ rho without one (event RESAMPLE).
 * Draws are keyed exactly as in decoding: key (seed, keys[i][0]), counter
 * (vocabulary block, keys[i][1] = the position being decided, event), so row i
 * reproduces the decision a decode step takes for a branch of sequence
 * keys[i][0] whose verification decides position keys[i][1].
 * ------------------------------------------------------------------------- */
typedef struct {
    int32_t vocab;           /* V, 1 .. 65536 */
    float temperature;       /* > 0 */
    float top_p;             /* (0, 1] */
    uint64_t seed;           /* Philox key word 0 */
    int32_t second_proposal; /* LOOPSPEC_SP_*; the ungated variants need has_second */
    int32_t has_second;      /* 0: single proposal (no d2 readout; z2 may be NULL) */
} loopspec_cascade_cfg;

/* Bytes of device workspace loopspec_cascade needs for `rows` rows of a
 * vocabulary: the barrier state of the shards of up to 64 rows in flight
 * (34880 bytes per row when a row spans several workgroups, none otherwise)
 * plus one error word.  0 for an invalid vocabulary or row count. */
uint64_t loopspec_cascade_workspace_bytes(int32_t vocab, int32_t rows);

/* Run the decisions of `rows` rows (device pointers, all on `stream`, a
 * hipStream_t; the call waits for the result).
 *   z1_dev, z2_dev, zR_dev: fp32 logits, row i at + i * z_stride
 *   keys_dev:  [rows][2] int32 (sequence, position being decided)
 *   out_dev:   [rows][6] int32: committed token, its source (1 first proposal,
 *              2 second, 0 resampled), x1, gate (1 when a second proposal was
 *              drawn), x2 (-1 without one), residuals met without positive mass
 *   q1_dev, q2_dev: [rows][vocab] fp32: the proposal distributions (q2 only
 *              where a second proposal was drawn)
 *   workspace_dev: caller-owned device memory of at least
 *              loopspec_cascade_workspace_bytes(vocab, rows) bytes; its
 *              contents on entry do not matter (the call clears it).
 * Calls that share a workspace must not overlap.  Errors: EINVAL (arguments,
 * workspace too small), EHIP (a launch failed or its shards' wait gave up),
 * ESTATE. */
int loopspec_cascade(const loopspec_cascade_cfg* cfg, int32_t rows, const float* z1_dev, const float* z2_dev,
                     const float* zR_dev, int64_t z_stride, const int32_t* keys_dev, int32_t* out_dev,
                     float* q1_dev, float* q2_dev, void* workspace_dev, uint64_t workspace_bytes, void* stream);

/* loopspec_cascade without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops, harnesses that
 * forbid hipMalloc): the same decisions, bit for bit, with the barrier state
 * kept in a static device array of the library (2.2 MiB: 64 rows in flight,
 * longer row lists run in launches of 64 rows) that each GPU holds until the
 * process ends.  Allocates nothing.  Every call on one GPU shares that GPU's
 * array, so calls that overlap on one GPU (other host threads, other streams)
 * race and must not be issued; consecutive calls are fine (each clears the
 * array first).  Arguments and errors as loopspec_cascade; ECAPACITY would
 * mean a row list the array cannot hold. */
int loopspec_cascade_noalloc(const loopspec_cascade_cfg* cfg, int32_t rows, const float* z1_dev,
                             const float* z2_dev, const float* zR_dev, int64_t z_stride, const int32_t* keys_dev,
                             int32_t* out_dev, float* q1_dev, float* q2_dev, void* stream);

/* Library version string. */
const char* loopspec_version(void);

#ifdef __cplusplus
}
#endif
#endif /* LOOPSPEC_H */
