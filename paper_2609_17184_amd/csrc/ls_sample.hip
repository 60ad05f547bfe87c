// Sampling readouts (temperature > 0), split over the vocabulary.
//
//  * readout distribution (Sec. 3.1: post-layers apply temperature, optional
//    top-p, softmax): p = softmax(z / T); top-p keeps token v iff the mass of
//    the tokens ranked strictly before it (descending p, ties by lower id) is
//    below top_p, then renormalises;
//  * depth d1: q1 = p_{d1} is kept in the branch's slot, x1 ~ q1 (early
//    drafting, Sec. 4.2);
//  * depth d2: the gate opens iff q2~(x1) < q1(x1) (Eq. adaptive-gate); then
//    q2 = q2~ (-) q1 (Eq. residual-proposal) is kept and x2 ~ q2; the
//    ablation's ungated variants (Table 3) always propose, from q2~ (-) q1 or
//    from q2~, with x1 masked out and the rest renormalised (no proposal when
//    nothing is left);
//  * depth R: cascade verification (Alg. 1, Verify): accept x1 iff
//    U1 < min(1, p(x1)/q1(x1)); else rho = p (-) q1 and, when the gate opened,
//    accept x2 iff U2 < min(1, rho(x2)/q2(x2)); else x ~ rho (-) q2 (or rho);
//  * vanilla decoding and the first token after prefill: x ~ p.
// (mu (-) nu) = [mu - nu]_+ / sum [mu - nu]_+ (Eq. residual-op); with no
// positive mass it returns mu and counts the event.
//
// Layout.  A row is split over NS workgroups (shards) of 256 threads, each
// thread holding E consecutive ids in registers from the logits load to the
// last decision, so a readout streams its logits once and every pass over the
// vocabulary runs on NS CUs.  The shards of a row meet at row barriers (an
// arrival counter per row, device-scope; a wait that does not end within the
// spin budget sets the error word and gives up, so a launch always ends).
// Before a barrier each shard publishes a few values (its maximum, its sum,
// its best race key, the owner's value of one id); after it every shard
// combines all shards' values in shard order, so every shard takes the same
// decisions and the combination order is fixed (run-to-run and batch
// invariant).  Probability masses that decide top-p cuts and residual
// normalisers are summed as 2^-40 fixed-point integers: integer sums do not
// depend on their order, and the cut is decided exactly on them.
//
// Top-p boundary without sorting: the kept set is {p > b} plus, in id order,
// ties at b while the mass before them stays below top_p, where b is the
// smallest probability whose strictly-greater mass is below top_p.  b is found
// by radix selection over the fp32 bit pattern (order-preserving for p >= 0):
// three rounds of 11, 10 and 10 bits, each a mass histogram of the candidates
// (the ids whose leading bits match the digits chosen so far), summed over the
// shards with integer atomics; the round's digit is the lowest non-empty bin
// whose mass above (everything beyond the bin) is still below top_p.
//
// Randomness: Philox4x64-10 (Salmon et al., SC'11), key = (seed, sequence),
// counter = (block, position of the token being decided, event, 0).  A
// categorical draw is an exponential race argmax_v w_v / -log U_v with U_v the
// word v % 4 of block v / 4 mapped to (0,1) by its top 23 bits plus one half;
// an accept test uses word 0 of block 0 mapped to [0,1) by its top 24 bits.
// The race is invariant to a positive scale of its weights, so a residual
// is raced unnormalised where its normaliser is not yet known.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/loopspec.h"
#include "ls_sample.h"

namespace ls {

enum Event { EV_TARGET = 1, EV_DRAFT1 = 2, EV_DRAFT2 = 3, EV_ACC1 = 4, EV_ACC2 = 5, EV_RESAMPLE = 6 };

// ---------------------------------------------------------------------------
// Philox4x64-10
// ---------------------------------------------------------------------------
struct P4 {
    unsigned long long x[4];
};

__device__ __forceinline__ P4 philox(unsigned long long c0, unsigned long long c1, unsigned long long c2,
                                     unsigned long long c3, unsigned long long k0, unsigned long long k1) {
    const unsigned long long M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const unsigned long long W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r) {
            k0 += W0;
            k1 += W1;
        }
        const unsigned long long hi0 = __umul64hi(M0, c0), lo0 = M0 * c0;
        const unsigned long long hi1 = __umul64hi(M1, c2), lo1 = M1 * c2;
        const unsigned long long n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
    }
    return P4{{c0, c1, c2, c3}};
}

__device__ __forceinline__ float u24(unsigned long long w) { return (float)(w >> 40) * (1.0f / 16777216.0f); }
__device__ __forceinline__ float u23_open(unsigned long long w) {
    return ((float)(w >> 41) + 0.5f) * (1.0f / 8388608.0f);
}
__device__ __forceinline__ float accept_u(unsigned long long seed, int seq, int pos, int ev) {
    return u24(philox(0ull, (unsigned long long)pos, (unsigned long long)ev, 0ull, seed, (unsigned long long)seq).x[0]);
}

// ---------------------------------------------------------------------------
// fixed point masses: p in [0, 1] as floor(p * 2^40); a histogram word packs
// (count << 44) | mass (the masses of a row sum to < 2^44, counts to < 2^20)
// ---------------------------------------------------------------------------
constexpr float kFix = 1099511627776.0f;   // 2^40
constexpr int kCountShift = 44;
constexpr unsigned long long kMassMask = (1ull << kCountShift) - 1;
__device__ __forceinline__ unsigned long long fix40(float p) { return (unsigned long long)(p * kFix); }
__device__ __forceinline__ float unfix40(unsigned long long m) { return (float)((double)m * (1.0 / 1099511627776.0)); }

// ---------------------------------------------------------------------------
// shard context and workgroup reductions (fixed order: a xor butterfly inside
// each wave, then the four waves in order)
// ---------------------------------------------------------------------------
// LDS of a shard: the histogram of a radix round; xu[0..3], xf, xi[0..3]
// the four waves' values of a reduction; xu[4..7], xi[4..7] single values;
// xu[16..31] the two banks of published values when the row has one shard
struct SLds {
    unsigned long long hist[1 << 11];
    unsigned long long xu[32];
    float xf[8];
    int xi[8];
};

struct SCtx {
    int V, E, NS, s, lo, hi;    // shard s of the row; this thread's ids [lo, hi)
    bool v4;                    // 16-byte accesses (V % 4 == 0)
    unsigned long long* rw;     // the row's scratch words (NS > 1)
    int nsync;                  // row barriers passed
    int32_t* err;
    SLds* l;
};

__device__ __forceinline__ unsigned long long shfl_xor_u64(unsigned long long v, int o) {
    const unsigned lo = __shfl_xor((unsigned)v, o), hi = __shfl_xor((unsigned)(v >> 32), o);
    return ((unsigned long long)hi << 32) | lo;
}
__device__ __forceinline__ unsigned long long shfl_down_u64(unsigned long long v, int o) {
    const unsigned lo = __shfl_down((unsigned)v, o), hi = __shfl_down((unsigned)(v >> 32), o);
    return ((unsigned long long)hi << 32) | lo;
}

__device__ __forceinline__ float wg_max(float v, SCtx& c) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    __syncthreads();
    if ((threadIdx.x & 63) == 0) c.l->xf[threadIdx.x >> 6] = v;
    __syncthreads();
    return fmaxf(fmaxf(c.l->xf[0], c.l->xf[1]), fmaxf(c.l->xf[2], c.l->xf[3]));
}
__device__ __forceinline__ float wg_sum(float v, SCtx& c) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) c.l->xf[threadIdx.x >> 6] = v;
    __syncthreads();
    return ((c.l->xf[0] + c.l->xf[1]) + c.l->xf[2]) + c.l->xf[3];
}
__device__ __forceinline__ unsigned long long wg_sum_u64(unsigned long long v, SCtx& c) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += shfl_xor_u64(v, o);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) c.l->xu[threadIdx.x >> 6] = v;
    __syncthreads();
    return c.l->xu[0] + c.l->xu[1] + c.l->xu[2] + c.l->xu[3];
}
__device__ __forceinline__ unsigned long long wg_max_u64(unsigned long long v, SCtx& c) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const unsigned long long w = shfl_xor_u64(v, o);
        v = w > v ? w : v;
    }
    __syncthreads();
    if ((threadIdx.x & 63) == 0) c.l->xu[threadIdx.x >> 6] = v;
    __syncthreads();
    unsigned long long m = c.l->xu[0];
    for (int k = 1; k < 4; ++k) m = c.l->xu[k] > m ? c.l->xu[k] : m;
    return m;
}
__device__ __forceinline__ int wg_min_i(int v, SCtx& c) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = min(v, __shfl_xor(v, o));
    __syncthreads();
    if ((threadIdx.x & 63) == 0) c.l->xi[threadIdx.x >> 6] = v;
    __syncthreads();
    return min(min(c.l->xi[0], c.l->xi[1]), min(c.l->xi[2], c.l->xi[3]));
}
// the value of the one thread that has it (own = true), else 0 (at most one owner)
__device__ __forceinline__ unsigned long long wg_owner_u64(bool own, unsigned long long v, SCtx& c) {
    return wg_sum_u64(own ? v : 0ull, c);
}

// ---------------------------------------------------------------------------
// row barriers and the values shards exchange across them
// ---------------------------------------------------------------------------
constexpr unsigned kSyncSpin = 1u << 18;

__device__ __forceinline__ void row_sync(SCtx& c) {
    c.nsync += 1;
    if (c.NS == 1) {
        __syncthreads();
        return;
    }
    __builtin_amdgcn_s_waitcnt(0);          // this thread's device-scope stores and atomics have completed
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long* cnt = c.rw + kRowCnt;
        __hip_atomic_fetch_add(cnt, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const unsigned long long target = (unsigned long long)c.NS * (unsigned long long)c.nsync;
        for (unsigned n = 0; __hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target; ++n) {
            if (n > kSyncSpin) {
                atomicOr(c.err, kErrPoll);
                break;
            }
            if ((n & 63) == 63 && (__hip_atomic_load(c.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & kErrPoll))
                break;
            __builtin_amdgcn_s_sleep(1);
        }
    }
    __syncthreads();
}

// slot k of this shard's partials for the coming barrier (a workgroup-uniform
// value; the banks alternate so no shard overwrites a value another shard may
// still be reading from the previous barrier)
__device__ __forceinline__ void publish(SCtx& c, int k, unsigned long long v) {
    if (c.NS == 1) {
        if (threadIdx.x == 0) c.l->xu[16 + (c.nsync & 1) * kPartSlots + k] = v;
        return;
    }
    if (threadIdx.x == 0) {
        unsigned long long* p = c.rw + kRowPart + ((c.nsync & 1) * kSShardsMax + c.s) * kPartSlots + k;
        __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}
__device__ __forceinline__ unsigned long long part(const SCtx& c, int s, int k) {
    if (c.NS == 1) return c.l->xu[16 + ((c.nsync - 1) & 1) * kPartSlots + k];
    const unsigned long long* p = c.rw + kRowPart + ((((c.nsync - 1) & 1) * kSShardsMax + s) * kPartSlots) + k;
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// after the barrier: the shards' values of slot k combined in shard order
__device__ __forceinline__ unsigned long long gather_sum(const SCtx& c, int k) {
    unsigned long long t = 0;
    for (int s = 0; s < c.NS; ++s) t += part(c, s, k);
    return t;
}
__device__ __forceinline__ unsigned long long gather_max(const SCtx& c, int k) {
    unsigned long long t = 0;
    for (int s = 0; s < c.NS; ++s) {
        const unsigned long long v = part(c, s, k);
        t = v > t ? v : t;
    }
    return t;
}

// Leaving the row: the last shard to arrive resets the barrier counter and the
// histograms (every other shard has read them), so the scratch is zero for the
// next launch.
__device__ __forceinline__ void row_exit(SCtx& c) {
    if (c.NS == 1) return;
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) {
        const unsigned long long old =
            __hip_atomic_fetch_add(c.rw + kRowCnt, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        c.l->xi[4] = old + 1 == (unsigned long long)c.NS * (unsigned long long)(c.nsync + 1);
    }
    __syncthreads();
    if (!c.l->xi[4]) return;
    for (int i = threadIdx.x; i < kHistWords; i += blockDim.x)
        __hip_atomic_store(c.rw + kRowHist + i, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (threadIdx.x == 0) __hip_atomic_store(c.rw + kRowCnt, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------------------
// per-thread vocabulary slices
// ---------------------------------------------------------------------------
template <int E>
__device__ __forceinline__ void load_row(const SCtx& c, const float* a, float (&v)[E], float fill) {
#pragma unroll
    for (int k = 0; k < E; k += 4) {
        const int id = c.lo + k;
        if (c.v4 && id < c.hi) {
            const float4 x = *(const float4*)(a + id);
            v[k] = x.x;
            v[k + 1] = x.y;
            v[k + 2] = x.z;
            v[k + 3] = x.w;
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[k + e] = id + e < c.hi ? a[id + e] : fill;
        }
    }
}
template <int E>
__device__ __forceinline__ void store_row(const SCtx& c, float* a, const float (&v)[E]) {
#pragma unroll
    for (int k = 0; k < E; k += 4) {
        const int id = c.lo + k;
        if (c.v4 && id < c.hi) {
            *(float4*)(a + id) = make_float4(v[k], v[k + 1], v[k + 2], v[k + 3]);
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (id + e < c.hi) a[id + e] = v[k + e];
        }
    }
}
__device__ __forceinline__ bool owns(const SCtx& c, int x) { return x >= c.lo && x < c.hi; }
// this thread's value at id x (x owned by it)
template <int E>
__device__ __forceinline__ float pick(const SCtx& c, const float (&v)[E], int x) {
    // a sum of products with 0/1 (a select chain the compiler would turn into a
    // dynamically indexed copy of the array in scratch memory)
    float r = 0.f;
#pragma unroll
    for (int k = 0; k < E; ++k) r = fmaf(v[k], c.lo + k == x ? 1.f : 0.f, r);
    return r;
}

// ---------------------------------------------------------------------------
// readout distribution
// ---------------------------------------------------------------------------
// Top-p filter of p (normalised softmax, in registers), exact on fixed-point masses.
template <int E>
__device__ __forceinline__ void topp_filter(SCtx& c, float (&p)[E], float top_p) {
    const unsigned long long Tfp = fix40(top_p);
    unsigned prefix = 0;               // leading bits chosen so far
    unsigned long long A = 0;          // mass strictly above the candidates
    unsigned long long nb_cnt = 0;     // candidates left at the last round (ties at b)
    unsigned long long* gh = c.NS > 1 ? c.rw + kRowHist : nullptr;
#pragma unroll
    for (int r = 0; r < 3; ++r) {
        const int bits = kRadixBits[r], shift = kRadixShift[r], nb = 1 << bits;
        for (int b = threadIdx.x; b < nb; b += blockDim.x) c.l->hist[b] = 0ull;
        __syncthreads();
#pragma unroll
        for (int k = 0; k < E; ++k) {
            if (c.lo + k >= c.hi) continue;
            const unsigned key = __float_as_uint(p[k]);
            if ((key >> (shift + bits)) != prefix) continue;
            atomicAdd(&c.l->hist[(key >> shift) & (nb - 1)], (1ull << kCountShift) | fix40(p[k]));
        }
        __syncthreads();
        if (c.NS > 1) {
            for (int b = threadIdx.x; b < nb; b += blockDim.x) {
                const unsigned long long v = c.l->hist[b];
                if (v) __hip_atomic_fetch_add(gh + b, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            row_sync(c);
            for (int b = threadIdx.x; b < nb; b += blockDim.x)
                c.l->hist[b] = __hip_atomic_load(gh + b, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __syncthreads();
            gh += nb;
        }
        // digit: the lowest non-empty bin j with A + (mass of bins above j) < top_p.
        // Thread t covers bins [t*B, t*B + B); suffix sums run from the top bin down.
        const int B = nb / kSThreads;
        unsigned long long local = 0;
        for (int q = 0; q < B; ++q) local += c.l->hist[threadIdx.x * B + q] & kMassMask;
        // exclusive suffix over threads: wave-inclusive suffix, then the waves above
        unsigned long long inc = local;
        const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const unsigned long long y = shfl_down_u64(inc, o);
            if (lane + o < 64) inc += y;
        }
        __syncthreads();
        if (lane == 0) c.l->xu[w] = inc;       // wave totals
        __syncthreads();
        unsigned long long above = inc - local;
        for (int ww = w + 1; ww < 4; ++ww) above += c.l->xu[ww];
        int cand = 0x7FFFFFFF;
        unsigned long long acand = 0;
        for (int q = B - 1; q >= 0; --q) {
            const int j = threadIdx.x * B + q;
            const unsigned long long h = c.l->hist[j];
            if ((h >> kCountShift) != 0 && A + above < Tfp) {
                cand = j;                          // lower bins of this thread come later and win
                acand = above;
            }
            above += h & kMassMask;
        }
        const int j = wg_min_i(cand, c);
        if (j == 0x7FFFFFFF) {                  // cannot happen: the top non-empty bin always qualifies
            if (threadIdx.x == 0) atomicOr(c.err, ERR_TREE);
            return;
        }
        // the owner of bin j publishes its mass above through LDS
        __syncthreads();
        if (cand == j) {
            c.l->xu[4] = acand;
            c.l->xu[5] = c.l->hist[j] >> kCountShift;
        }
        __syncthreads();
        A += c.l->xu[4];
        nb_cnt = c.l->xu[5];
        prefix = (prefix << bits) | (unsigned)j;
        __syncthreads();
    }
    // b = the boundary probability; A = mass of {p > b}; nb_cnt ties at b
    const float b = __uint_as_float(prefix);
    const unsigned long long bfp = fix40(b);
    unsigned long long kt;                     // ties kept (the first ones in id order)
    if (A >= Tfp)
        kt = 0;
    else if (bfp == 0)
        kt = nb_cnt;
    else
        kt = min(nb_cnt, (Tfp - A + bfp - 1) / bfp);
    // ranks of the ties, only when some are dropped
    long long rank0 = 0;
    int mine = 0;
#pragma unroll
    for (int k = 0; k < E; ++k)
        if (c.lo + k < c.hi && __float_as_uint(p[k]) == prefix) ++mine;
    if (kt < nb_cnt) {
        // exclusive prefix of tie counts over this shard's threads, then over shards
        int inc = mine;
        const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int y = __shfl_up(inc, o);
            if (lane >= o) inc += y;
        }
        __syncthreads();
        if (lane == 63) c.l->xi[w] = inc;
        __syncthreads();
        rank0 = inc - mine;
        for (int ww = 0; ww < w; ++ww) rank0 += c.l->xi[ww];
        const int shard_ties = c.l->xi[0] + c.l->xi[1] + c.l->xi[2] + c.l->xi[3];
        publish(c, 0, (unsigned long long)shard_ties);
        row_sync(c);
        for (int s = 0; s < c.s; ++s) rank0 += (long long)part(c, s, 0);
    }
    const unsigned long long K = A + kt * bfp;  // kept mass
    const float inv = (float)(1099511627776.0 / (double)K);
    long long rk = rank0;
#pragma unroll
    for (int k = 0; k < E; ++k) {
        const unsigned key = __float_as_uint(p[k]);
        bool keep = key > prefix;
        if (key == prefix && c.lo + k < c.hi) {
            keep = rk < (long long)kt;
            ++rk;
        }
        p[k] = keep ? p[k] * inv : 0.f;
    }
}

// p = readout distribution of logits z: softmax(z / T), then top-p.  The
// shards' (max, sum of exp) pairs combine in shard order.
template <int E>
__device__ __forceinline__ void shard_dist(SCtx& c, const float* z, float T, float top_p, float (&p)[E]) {
    load_row(c, z, p, -INFINITY);
    float mx = -INFINITY;
#pragma unroll
    for (int k = 0; k < E; ++k) {
        p[k] = c.lo + k < c.hi ? p[k] / T : -INFINITY;
        mx = fmaxf(mx, p[k]);
    }
    const float m = wg_max(mx, c);
    float se = 0.f;
#pragma unroll
    for (int k = 0; k < E; ++k)
        if (c.lo + k < c.hi) se += expf(p[k] - m);
    const float l = wg_sum(se, c);
    publish(c, 0, __float_as_uint(m));
    publish(c, 1, __float_as_uint(l));
    row_sync(c);
    float M = -INFINITY;
    for (int s = 0; s < c.NS; ++s) M = fmaxf(M, __uint_as_float((unsigned)part(c, s, 0)));
    float Z = 0.f;
    for (int s = 0; s < c.NS; ++s) {
        const float ms = __uint_as_float((unsigned)part(c, s, 0)), ls = __uint_as_float((unsigned)part(c, s, 1));
        if (ms > -INFINITY) Z += ls * expf(ms - M);
    }
    const float invZ = 1.0f / Z;
#pragma unroll
    for (int k = 0; k < E; ++k) {
        p[k] = c.lo + k < c.hi ? expf(p[k] - M) * invZ : 0.f;
    }
    if (top_p < 1.0f) topp_filter(c, p, top_p);
}

// this shard's best exponential-race key over weights w >= 0 (w = 0 never
// wins): (race value bits << 32) | (0xFFFFFFFF - id), so the maximum key is the
// largest value with ties to the lowest id; 0 when no weight is positive
template <int E>
__device__ __forceinline__ unsigned long long race_key(SCtx& c, const float (&w)[E], unsigned long long seed, int seq, int pos,
                                       int ev) {
    unsigned long long best = 0;
#pragma unroll
    for (int k = 0; k < E; k += 4) {
        const int v0 = c.lo + k;
        if (v0 >= c.hi) continue;
        const P4 r = philox((unsigned long long)(v0 >> 2), (unsigned long long)pos, (unsigned long long)ev, 0ull,
                            seed, (unsigned long long)seq);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int v = v0 + e;
            if (v >= c.hi || !(w[k + e] > 0.f)) continue;
            const float sc = w[k + e] / -logf(u23_open(r.x[e]));
            const unsigned long long key = ((unsigned long long)__float_as_uint(sc) << 32) | (0xFFFFFFFFu - (unsigned)v);
            best = key > best ? key : best;
        }
    }
    return wg_max_u64(best, c);
}
__device__ __forceinline__ int key_token(unsigned long long key) {
    return key ? (int)(0xFFFFFFFFu - (unsigned)(key & 0xFFFFFFFFull)) : -1;
}
// a categorical draw over w (one barrier)
template <int E>
__device__ __forceinline__ int race(SCtx& c, const float (&w)[E], unsigned long long seed, int seq, int pos, int ev) {
    publish(c, 0, race_key(c, w, seed, seq, pos, ev));
    row_sync(c);
    return key_token(gather_max(c, 0));
}

// ---------------------------------------------------------------------------
// one readout row
// ---------------------------------------------------------------------------
enum Role { ROLE_NONE = 0, ROLE_TARGET = 1, ROLE_DRAFT1 = 2, ROLE_DRAFT2 = 3, ROLE_VERIFY = 4 };

struct SampleCfg {
    float T, top_p;
    int variant;                 // LOOPSPEC_SP_*
    unsigned long long seed;
};

struct RowJob {
    int role;
    const float* z;              // readout logits [V]
    float* q1;                   // DRAFT1: written; DRAFT2, VERIFY: read
    float* q2;                   // DRAFT2: written; VERIFY: read
    float* q2t;                  // DRAFT2: the readout at d2 written; VERIFY: read (NULL: not kept)
    int x1, gate, x2;            // DRAFT2: x1; VERIFY: x1, gate, x2
    int seq, pos;                // key word and position being decided
};

struct RowOut {
    int tok, aux, zero_mass, bad;
    int has_tv;                      // VERIFY: TV(p, q1) and TV(p, q2~) below (2^-40 units)
    unsigned long long tv1, tv2;
};

template <int E>
__device__ __forceinline__ RowOut sample_row(SCtx& c, const SampleCfg& cfg, const RowJob& j) {
    RowOut o{-1, 0, 0, 0, 0, 0ull, 0ull};
    if (j.role == ROLE_NONE) return o;
    const int V = c.V;
    float p[E];
    shard_dist(c, j.z, cfg.T, cfg.top_p, p);
    if (j.role == ROLE_TARGET) {
        o.tok = race(c, p, cfg.seed, j.seq, j.pos, EV_TARGET);
        return o;
    }
    if (j.role == ROLE_DRAFT1) {
        store_row(c, j.q1, p);
        o.tok = race(c, p, cfg.seed, j.seq, j.pos, EV_DRAFT1);
        return o;
    }
    const int x1 = j.x1;
    if (x1 < 0 || x1 >= V) {     // no first draft recorded: an inconsistent tree
        o.bad = 1;
        if (j.role == ROLE_VERIFY) o.tok = race(c, p, cfg.seed, j.seq, j.pos, EV_RESAMPLE);
        return o;
    }
    float q1[E], r[E];
    load_row(c, j.q1, q1, 0.f);
    unsigned long long sr = 0, sp = 0;
#pragma unroll
    for (int k = 0; k < E; ++k) {
        r[k] = fmaxf(p[k] - q1[k], 0.f);
        sr += fix40(r[k]);
        sp += fix40(p[k]);
    }
    const bool own1 = owns(c, x1);
    if (j.role == ROLE_DRAFT2) {
        if (j.q2t) store_row(c, j.q2t, p);       // q2~, for TV(p_R, p_d2) at verification
        // one barrier: sums of [p - q1]_+ and of p, and the owner's values at x1
        const unsigned long long S = wg_sum_u64(sr, c), P = wg_sum_u64(sp, c);
        const unsigned long long px1 = wg_owner_u64(own1, __float_as_uint(pick(c, p, x1)), c);
        const unsigned long long rx1 = wg_owner_u64(own1, fix40(pick(c, r, x1)), c);
        const unsigned long long px1f = wg_owner_u64(own1, fix40(pick(c, p, x1)), c);
        publish(c, 0, S);
        publish(c, 1, P);
        publish(c, 2, px1);
        publish(c, 3, rx1);
        publish(c, 4, px1f);
        row_sync(c);
        const unsigned long long gS = gather_sum(c, 0), gP = gather_sum(c, 1);
        const float gpx1 = __uint_as_float((unsigned)gather_sum(c, 2));
        const unsigned long long grx1 = gather_sum(c, 3), gpx1f = gather_sum(c, 4);
        bool open;
        float q2[E];
        if (cfg.variant == LOOPSPEC_SP_GATED) {
            open = gpx1 < j.q1[x1];                  // q2~(x1) < q1(x1)
            if (open) {
                const bool zm = gS == 0;
                o.zero_mass = zm;
                const float inv = zm ? 1.f : 1.0f / unfix40(gS);
#pragma unroll
                for (int k = 0; k < E; ++k) q2[k] = zm ? p[k] : r[k] * inv;
            }
        } else {
            // ungated: the base distribution with x1 masked out, renormalised
            const bool resid = cfg.variant == LOOPSPEC_SP_RESIDUAL;
            const bool zm = resid && gS == 0;        // q2~ (-) q1 without positive mass returns q2~
            const bool usep = !resid || zm;
            const unsigned long long left = usep ? gP - gpx1f : gS - grx1;
            open = left > 0;
            o.zero_mass = open && zm;
            const float inv = open ? 1.0f / unfix40(left) : 0.f;
#pragma unroll
            for (int k = 0; k < E; ++k)
                q2[k] = (c.lo + k == x1) ? 0.f : (usep ? p[k] : r[k]) * inv;
        }
        if (open) {
            store_row(c, j.q2, q2);
            o.tok = race(c, q2, cfg.seed, j.seq, j.pos, EV_DRAFT2);
            o.aux = o.tok >= 0;
        }
        return o;
    }
    // ---- ROLE_VERIFY: the cascade over the proposals --------------------------
    const bool gate = j.gate && j.x2 >= 0 && j.x2 < V;
    const int x2 = gate ? j.x2 : -1;
    const bool own2 = gate && owns(c, x2);
    const unsigned long long S1 = wg_sum_u64(sr, c);
    const unsigned long long px1 = wg_owner_u64(own1, __float_as_uint(pick(c, p, x1)), c);
    publish(c, 0, S1);
    publish(c, 1, px1);
    if (j.q2t) {
        // TV(p, q2~) = sum [p - q2~]_+ (both normalised), for the depth planner
        float t2[E];
        load_row(c, j.q2t, t2, 0.f);
        unsigned long long s2t = 0;
#pragma unroll
        for (int k = 0; k < E; ++k) s2t += fix40(fmaxf(p[k] - t2[k], 0.f));
        publish(c, 6, wg_sum_u64(s2t, c));
    }
    if (gate) {
        publish(c, 2, wg_owner_u64(own2, __float_as_uint(pick(c, r, x2)), c));
        publish(c, 3, wg_owner_u64(own2, __float_as_uint(pick(c, p, x2)), c));
    } else {
        // without a second proposal a rejection resamples from rho1: race
        // [p - q1]_+ now (and p, in case it has no positive mass)
        publish(c, 4, race_key(c, r, cfg.seed, j.seq, j.pos, EV_RESAMPLE));
        publish(c, 5, race_key(c, p, cfg.seed, j.seq, j.pos, EV_RESAMPLE));
    }
    row_sync(c);
    const unsigned long long gS1 = gather_sum(c, 0);
    const float gpx1 = __uint_as_float((unsigned)gather_sum(c, 1));
    o.has_tv = 1;
    o.tv1 = gS1;                                 // sum [p - q1]_+ = TV(p, q1)
    o.tv2 = j.q2t ? gather_sum(c, 6) : 0ull;
    const float u1 = accept_u(cfg.seed, j.seq, j.pos, EV_ACC1);
    if (u1 < fminf(1.0f, gpx1 / j.q1[x1])) {
        o.tok = x1;
        o.aux = 1;
        return o;
    }
    const bool zm1 = gS1 == 0;                   // rho1 = p (-) q1 without positive mass: p
    o.zero_mass = zm1;
    if (!gate) {
        o.tok = key_token(zm1 ? gather_max(c, 5) : gather_max(c, 4));
        return o;
    }
    const float invS1 = zm1 ? 1.f : 1.0f / unfix40(gS1);
    const float rho_x2 = zm1 ? __uint_as_float((unsigned)gather_sum(c, 3))
                             : __uint_as_float((unsigned)gather_sum(c, 2)) * invS1;
    const float u2 = accept_u(cfg.seed, j.seq, j.pos, EV_ACC2);
    if (u2 < fminf(1.0f, rho_x2 / j.q2[x2])) {
        o.tok = x2;
        o.aux = 2;
        return o;
    }
    // rho2 = rho1 (-) q2, raced unnormalised; rho1 itself if it has no positive mass
    float w[E];
    load_row(c, j.q2, w, 0.f);
    unsigned long long s2 = 0;
#pragma unroll
    for (int k = 0; k < E; ++k) {
        w[k] = fmaxf((zm1 ? p[k] : r[k] * invS1) - w[k], 0.f);     // [rho1 - q2]_+
        s2 += fix40(w[k]);
    }
    publish(c, 0, wg_sum_u64(s2, c));
    publish(c, 1, race_key(c, w, cfg.seed, j.seq, j.pos, EV_RESAMPLE));
#pragma unroll
    for (int k = 0; k < E; ++k) w[k] = zm1 ? p[k] : r[k] * invS1;   // rho1
    publish(c, 2, race_key(c, w, cfg.seed, j.seq, j.pos, EV_RESAMPLE));
    row_sync(c);
    const bool zm2 = gather_sum(c, 0) == 0;
    o.zero_mass += zm2;
    o.tok = key_token(zm2 ? gather_max(c, 2) : gather_max(c, 1));
    return o;
}

__device__ __forceinline__ SCtx make_ctx(const SGeo& g, int shard, unsigned long long* rw, int32_t* err, SLds* l) {
    SCtx c;
    c.V = g.V;
    c.E = g.E;
    c.NS = g.NS;
    c.s = shard;
    c.lo = min(g.V, shard * g.chunk + (int)threadIdx.x * g.E);
    c.hi = min(g.V, c.lo + g.E);
    c.v4 = (g.V & 3) == 0;
    c.rw = rw;
    c.nsync = 0;
    c.err = err;
    c.l = l;
    return c;
}

// ---------------------------------------------------------------------------
// decode steps: every readout row of the step (grid: rows_cap x NS shards)
// ---------------------------------------------------------------------------
template <int E>
__global__ void __launch_bounds__(kSThreads) k_finalize_sample(Sched s, int fin_op, const float* logits) {
    const SGeo g = sample_geo(s.g.V);
    const int i = blockIdx.x / g.NS, shard = blockIdx.x - i * g.NS;
    if (i >= *s.nC) return;
    __shared__ SLds lds;
    SCtx c = make_ctx(g, shard, s.srow + (size_t)i * kRowWords, s.err, &lds);
    const Row row = s.rowsC[i];
    const int b = row.slot, mode = *s.mode;
    RowJob j{};
    j.z = logits + (size_t)i * g.V;
    j.seq = row.seq;
    j.pos = row.pos + 1;
    j.x1 = j.x2 = -1;
    if (fin_op == FIN_TARGET || mode == MODE_VANILLA || mode == MODE_FORCED) {
        j.role = (fin_op == FIN_TARGET || row.depth == s.R) ? ROLE_TARGET : ROLE_NONE;
    } else if (row.depth == s.d1) {
        j.role = ROLE_DRAFT1;
        j.q1 = s.q1 + (size_t)b * g.V;
    } else if (s.d2 > 0 && row.depth == s.d2) {
        j.role = ROLE_DRAFT2;
        j.q1 = s.q1 + (size_t)b * g.V;
        j.q2 = s.q2 + (size_t)b * g.V;
        j.q2t = s.q2t + (size_t)b * g.V;
        j.x1 = s.s_x1[b];
    } else if (row.depth == s.R) {
        j.role = ROLE_VERIFY;
        j.q1 = s.q1 + (size_t)b * g.V;
        j.q2 = s.q2 + (size_t)b * g.V;
        j.q2t = s.d2 > 0 ? s.q2t + (size_t)b * g.V : nullptr;
        j.x1 = s.s_x1[b];
        j.gate = s.s_gate[b];
        j.x2 = s.s_x2[b];
    } else {
        j.role = ROLE_NONE;
    }
    const SampleCfg cfg{s.temperature, s.top_p, s.variant, *s.seed};
    const RowOut o = sample_row<E>(c, cfg, j);
    if (shard == 0 && threadIdx.x == 0) {
        s.ro_tok[i] = o.tok;
        s.ro_aux[i] = o.aux;
        if (o.zero_mass) atomicAdd((unsigned long long*)&s.stats[ST_ZERO_MASS], (unsigned long long)o.zero_mass);
        if (o.bad) atomicOr(s.err, ERR_TREE);
        if (o.has_tv) {                          // 2^-40 -> 2^-32 units
            atomicAdd((unsigned long long*)&s.stats[ST_TV1], o.tv1 >> 8);
            atomicAdd((unsigned long long*)&s.stats[ST_TV2], o.tv2 >> 8);
            atomicAdd((unsigned long long*)&s.stats[ST_TVN], 1ull);
        }
    }
    row_exit(c);
}

hipError_t launch_finalize_sample(const Sched& s, int fin_op, const float* logits, int rows_cap, hipStream_t st) {
    const SGeo g = sample_geo(s.g.V);
    const dim3 grid(rows_cap * g.NS), blk(kSThreads);
    switch (g.E) {
        case 4: hipLaunchKernelGGL(k_finalize_sample<4>, grid, blk, 0, st, s, fin_op, logits); break;
        case 8: hipLaunchKernelGGL(k_finalize_sample<8>, grid, blk, 0, st, s, fin_op, logits); break;
        case 12: hipLaunchKernelGGL(k_finalize_sample<12>, grid, blk, 0, st, s, fin_op, logits); break;
        case 16: hipLaunchKernelGGL(k_finalize_sample<16>, grid, blk, 0, st, s, fin_op, logits); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// Rows whose shards can all be resident at once (every shard of a row waits
// for the others at the row barriers): CUs x workgroups per CU / shards.
int sample_rows_resident(int V) {
    const SGeo g = sample_geo(V);
    const void* f = nullptr;
    switch (g.E) {
        case 4: f = (const void*)k_finalize_sample<4>; break;
        case 8: f = (const void*)k_finalize_sample<8>; break;
        case 12: f = (const void*)k_finalize_sample<12>; break;
        case 16: f = (const void*)k_finalize_sample<16>; break;
        default: return 0;
    }
    int dev = 0, cus = 0, per = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, f, kSThreads, 0) != hipSuccess) {
        (void)hipGetLastError();
        return 0;
    }
    return cus * per / g.NS;
}

__global__ void __launch_bounds__(256) k_zero_words(unsigned long long* p, size_t n) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = 0ull;
}

hipError_t launch_zero_words(unsigned long long* p, size_t n, hipStream_t st) {
    if (!n) return hipSuccess;
    const int blocks = (int)std::min<size_t>((n + 255) / 256, 1024);
    hipLaunchKernelGGL(k_zero_words, dim3(blocks), dim3(256), 0, st, p, n);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// standalone cascade over independent keyed positions (one launch per role)
// ---------------------------------------------------------------------------
struct CascadeArgs {
    int rows, row0;
    const float* z;              // logits of this role's depth, row i at z + i * zstride
    long long zstride;
    float *q1, *q2;              // [rows][V]
    const int32_t* keys;         // [rows][2]: sequence, position
    int32_t* out;                // [rows][6]: token, source, x1, gate, x2, zero-mass events
    unsigned long long* scratch; // kRowWords per row of the launch (row - row0), NS > 1
    int32_t* err;
    int vec;                     // 16-byte accesses allowed (rows and pointers 16-byte aligned)
};

template <int E>
__global__ void __launch_bounds__(kSThreads) k_cascade(SampleCfg cfg, CascadeArgs a, int role, int V) {
    const SGeo g = sample_geo(V);
    const int li = blockIdx.x / g.NS, shard = blockIdx.x - li * g.NS;
    const int i = a.row0 + li;
    if (i >= a.rows) return;
    __shared__ SLds lds;
    SCtx c = make_ctx(g, shard, g.NS > 1 ? a.scratch + (size_t)li * kRowWords : nullptr, a.err, &lds);
    c.v4 = c.v4 && a.vec;
    int32_t* o = a.out + (size_t)i * 6;
    RowJob j{};
    j.role = role;
    j.z = a.z + (size_t)i * a.zstride;
    j.q1 = a.q1 + (size_t)i * V;
    j.q2 = a.q2 + (size_t)i * V;
    j.seq = a.keys[2 * i];
    j.pos = a.keys[2 * i + 1];
    j.x1 = role == ROLE_DRAFT1 ? -1 : o[2];
    j.gate = o[3];
    j.x2 = o[4];
    const RowOut r = sample_row<E>(c, cfg, j);
    if (shard == 0 && threadIdx.x == 0) {
        if (role == ROLE_DRAFT1) {
            o[2] = r.tok;
            o[3] = 0;
            o[4] = -1;
            o[5] = r.zero_mass;
        } else if (role == ROLE_DRAFT2) {
            o[3] = r.aux;
            o[4] = r.aux ? r.tok : -1;
            o[5] += r.zero_mass;
        } else {
            o[0] = r.tok;
            o[1] = r.aux;
            o[5] += r.zero_mass;
        }
        if (r.bad) atomicOr(a.err, ERR_TREE);
    }
    row_exit(c);
}

}  // namespace ls

// ===========================================================================
// C ABI of the standalone cascade
// ===========================================================================
using namespace ls;

namespace {

// Scratch of the allocation-free entry point: the barrier state of
// kCascadeRowsPerLaunch rows (2.2 MiB) plus the launch's error word.  Each GPU
// holds its own copy until the process ends; host code reaches it only
// through the address hipGetSymbolAddress returns on that device.
constexpr size_t kScratchWords = (size_t)kCascadeRowsPerLaunch * kRowWords + 8;
static __device__ __align__(256) unsigned long long scratch[kScratchWords];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
unsigned long long* g_scratch_ptr[kMaxDevices] = {};

int scratch_ptr(unsigned long long** out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return LOOPSPEC_EHIP;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
            (void)hipGetLastError();
            return LOOPSPEC_EHIP;
        }
        g_scratch_ptr[dev] = (unsigned long long*)p;
    }
    *out = g_scratch_ptr[dev];
    return LOOPSPEC_OK;
}

int cascade_check(const loopspec_cascade_cfg* cfg, int32_t rows, const float* z1, const float* z2, const float* zR,
                  int64_t zstride, const int32_t* keys, int32_t* out, float* q1, float* q2) {
    if (!cfg || rows < 0 || !z1 || !zR || !keys || !out || !q1 || !q2) return LOOPSPEC_EINVAL;
    if (cfg->has_second && !z2) return LOOPSPEC_EINVAL;
    if (cfg->vocab < 1 || cfg->vocab > kSampleMaxVocab) return LOOPSPEC_EINVAL;
    if (!(cfg->temperature > 0.f) || !(cfg->top_p > 0.f && cfg->top_p <= 1.f)) return LOOPSPEC_EINVAL;
    if (cfg->second_proposal < LOOPSPEC_SP_GATED || cfg->second_proposal > LOOPSPEC_SP_NAIVE) return LOOPSPEC_EINVAL;
    if (cfg->second_proposal != LOOPSPEC_SP_GATED && !cfg->has_second) return LOOPSPEC_EINVAL;
    if (zstride < 0) return LOOPSPEC_EINVAL;
    return LOOPSPEC_OK;
}

// The three roles over every row, in launches of kCascadeRowsPerLaunch rows
// when a row takes several shards.  `rw` holds kRowWords per row of a launch
// and one more word for the error flag.
int cascade_run(const loopspec_cascade_cfg* cfg, int32_t rows, const float* z1, const float* z2, const float* zR,
                int64_t zstride, const int32_t* keys, int32_t* out, float* q1, float* q2, unsigned long long* rw,
                hipStream_t st) {
    if (!rows) return LOOPSPEC_OK;
    const SGeo g = sample_geo(cfg->vocab);
    const int per = g.NS > 1 ? kCascadeRowsPerLaunch : rows;
    if (g.NS > 1 && sample_rows_resident(cfg->vocab) < kCascadeRowsPerLaunch) return LOOPSPEC_EHIP;
    const size_t words = g.NS > 1 ? (size_t)std::min(rows, per) * kRowWords : 0;
    int32_t* err = (int32_t*)(rw + words);
    // barrier state and the error word start at zero (a fill kernel, not a memset)
    if (launch_zero_words(rw, words + 1, st) != hipSuccess) return LOOPSPEC_EHIP;
    SampleCfg sc{cfg->temperature, cfg->top_p, cfg->second_proposal, (unsigned long long)cfg->seed};
    CascadeArgs a{};
    a.rows = rows;
    a.zstride = zstride;
    a.q1 = q1;
    a.q2 = q2;
    a.keys = keys;
    a.out = out;
    a.scratch = rw;
    a.err = err;
    auto al = [](const void* q) { return ((uintptr_t)q & 15) == 0; };
    a.vec = (zstride & 3) == 0 && al(z1) && al(zR) && (!z2 || al(z2)) && al(q1) && al(q2);
    const int roles[3] = {ROLE_DRAFT1, ROLE_DRAFT2, ROLE_VERIFY};
    const float* zs[3] = {z1, z2, zR};
    for (int r0 = 0; r0 < rows; r0 += per) {
        const int n = std::min(per, rows - r0);
        a.row0 = r0;
        for (int k = 0; k < 3; ++k) {
            if (roles[k] == ROLE_DRAFT2 && !cfg->has_second) continue;
            a.z = zs[k];
            const dim3 grid(n * g.NS), blk(kSThreads);
            switch (g.E) {
                case 4: hipLaunchKernelGGL(k_cascade<4>, grid, blk, 0, st, sc, a, roles[k], cfg->vocab); break;
                case 8: hipLaunchKernelGGL(k_cascade<8>, grid, blk, 0, st, sc, a, roles[k], cfg->vocab); break;
                case 12: hipLaunchKernelGGL(k_cascade<12>, grid, blk, 0, st, sc, a, roles[k], cfg->vocab); break;
                case 16: hipLaunchKernelGGL(k_cascade<16>, grid, blk, 0, st, sc, a, roles[k], cfg->vocab); break;
                default: return LOOPSPEC_EINVAL;
            }
            if (hipGetLastError() != hipSuccess) return LOOPSPEC_EHIP;
        }
    }
    int32_t e = 0;
    if (hipMemcpyAsync(&e, err, 4, hipMemcpyDeviceToHost, st) != hipSuccess || hipStreamSynchronize(st) != hipSuccess)
        return LOOPSPEC_EHIP;
    if (e & kErrPoll) return LOOPSPEC_EHIP;
    if (e & ERR_TREE) return LOOPSPEC_ESTATE;
    return LOOPSPEC_OK;
}

}  // namespace

extern "C" {

uint64_t loopspec_cascade_workspace_bytes(int32_t vocab, int32_t rows) {
    if (vocab < 1 || vocab > kSampleMaxVocab || rows < 0) return 0;
    const SGeo g = sample_geo(vocab);
    const size_t per = g.NS > 1 ? (size_t)std::min(rows, kCascadeRowsPerLaunch) * kRowWords : 0;
    return (per + 1) * 8;
}

int loopspec_cascade(const loopspec_cascade_cfg* cfg, int32_t rows, const float* z1_dev, const float* z2_dev,
                     const float* zR_dev, int64_t z_stride, const int32_t* keys_dev, int32_t* out_dev, float* q1_dev,
                     float* q2_dev, void* workspace_dev, uint64_t workspace_bytes, void* stream) {
    int r = cascade_check(cfg, rows, z1_dev, z2_dev, zR_dev, z_stride, keys_dev, out_dev, q1_dev, q2_dev);
    if (r) return r;
    if (!workspace_dev || workspace_bytes < loopspec_cascade_workspace_bytes(cfg->vocab, rows)) return LOOPSPEC_EINVAL;
    return cascade_run(cfg, rows, z1_dev, z2_dev, zR_dev, z_stride, keys_dev, out_dev, q1_dev, q2_dev,
                       (unsigned long long*)workspace_dev, (hipStream_t)stream);
}

int loopspec_cascade_noalloc(const loopspec_cascade_cfg* cfg, int32_t rows, const float* z1_dev,
                             const float* z2_dev, const float* zR_dev, int64_t z_stride, const int32_t* keys_dev,
                             int32_t* out_dev, float* q1_dev, float* q2_dev, void* stream) {
    int r = cascade_check(cfg, rows, z1_dev, z2_dev, zR_dev, z_stride, keys_dev, out_dev, q1_dev, q2_dev);
    if (r) return r;
    if (loopspec_cascade_workspace_bytes(cfg->vocab, rows) > kScratchWords * 8) return LOOPSPEC_ECAPACITY;
    unsigned long long* p = nullptr;
    if ((r = scratch_ptr(&p))) return r;
    return cascade_run(cfg, rows, z1_dev, z2_dev, zR_dev, z_stride, keys_dev, out_dev, q1_dev, q2_dev, p,
                       (hipStream_t)stream);
}

}  // extern "C"
