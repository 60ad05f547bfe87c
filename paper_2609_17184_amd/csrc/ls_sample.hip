// Sampling readouts (temperature > 0): one workgroup per readout row.
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
// Randomness: Philox4x64-10 (Salmon et al., SC'11), key = (seed, sequence),
// counter = (block, position of the token being decided, event, 0).  A
// categorical draw is an exponential race argmax_v w_v / -log U_v with U_v the
// word v % 4 of block v / 4 mapped to (0,1) by its top 23 bits plus one half;
// an accept test uses word 0 of block 0 mapped to [0,1) by its top 24 bits.
#include "ls_sched.h"

namespace ls {

enum Event { EV_TARGET = 1, EV_DRAFT1 = 2, EV_DRAFT2 = 3, EV_ACC1 = 4, EV_ACC2 = 5, EV_RESAMPLE = 6 };

constexpr int kThreads = 1024;

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

// ---------------------------------------------------------------------------
// deterministic block reductions: per-thread values combine by a fixed
// xor-butterfly inside each wave, then in wave order
// ---------------------------------------------------------------------------
struct Red {
    float* f;      // [32]
    int* i;        // [32]
};

__device__ float block_sum(float v, Red r) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) r.f[w] = v;
    __syncthreads();
    float s = 0.f;
    for (int k = 0; k < nw; ++k) s += r.f[k];
    return s;
}

__device__ float block_max(float v, Red r) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) r.f[w] = v;
    __syncthreads();
    float s = -INFINITY;
    for (int k = 0; k < nw; ++k) s = fmaxf(s, r.f[k]);
    return s;
}

__device__ __forceinline__ bool beats(float v, int i, float bv, int bi) {
    return bi < 0 || v > bv || (v == bv && i < bi);
}

// arg-max with ties to the lowest id; (-inf, -1) when every value is -inf
__device__ int block_argmax(float v, int id, Red r) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const float ov = __shfl_xor(v, o);
        const int oi = __shfl_xor(id, o);
        if (oi >= 0 && beats(ov, oi, v, id)) {
            v = ov;
            id = oi;
        }
    }
    const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) {
        r.f[w] = v;
        r.i[w] = id;
    }
    __syncthreads();
    float bv = -INFINITY;
    int bi = -1;
    for (int k = 0; k < nw; ++k)
        if (r.i[k] >= 0 && beats(r.f[k], r.i[k], bv, bi)) {
            bv = r.f[k];
            bi = r.i[k];
        }
    return bi;
}

// ---------------------------------------------------------------------------
// per-row helpers; thread t owns the contiguous ids [t*E, min(V, (t+1)*E))
// ---------------------------------------------------------------------------
struct Ctx {
    int V, E, lo, hi;
    Red red;
};

// A thread's ids are contiguous: when every slice is a whole number of
// 4-id groups the passes over global arrays read and write 16 bytes per id
// group (a quarter of the memory requests of 4-byte accesses).
__device__ __forceinline__ bool vec4(const Ctx& c) { return ((c.E | c.V) & 3) == 0; }
__device__ __forceinline__ float4 ld4(const float* a, int v) { return *(const float4*)(a + v); }
__device__ __forceinline__ void st4(float* a, int v, float4 x) { *(float4*)(a + v) = x; }
__device__ __forceinline__ float get4(const float4& x, int e) { return e == 0 ? x.x : e == 1 ? x.y : e == 2 ? x.z : x.w; }

// p = readout distribution of logits z (temperature, softmax, top-p).  A
// thread's ids stay in registers through every pass (the top-p threshold
// search alone makes about thirty), and p is written once at the end.
constexpr int kEMax = kSampleMaxVocab / kThreads;   // ids per thread
__device__ void readout_dist(const Ctx& c, const float* z, float* p, float T, float top_p) {
    float pr[kEMax];
    float mx = -INFINITY;
    if (vec4(c)) {
#pragma unroll
        for (int k = 0; k < kEMax; k += 4) {
            float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
            if (c.lo + k < c.hi) a = ld4(z, c.lo + k);
            pr[k] = a.x / T;
            pr[k + 1] = a.y / T;
            pr[k + 2] = a.z / T;
            pr[k + 3] = a.w / T;
        }
    } else {
#pragma unroll
        for (int k = 0; k < kEMax; ++k) pr[k] = c.lo + k < c.hi ? z[c.lo + k] / T : 0.f;
    }
#pragma unroll
    for (int k = 0; k < kEMax; ++k)
        if (c.lo + k < c.hi) mx = fmaxf(mx, pr[k]);
    mx = block_max(mx, c.red);
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < kEMax; ++k) {
        if (c.lo + k < c.hi) {
            const float e = expf(pr[k] - mx);
            pr[k] = e;
            s += e;
        } else {
            pr[k] = 0.f;
        }
    }
    s = block_sum(s, c.red);
    const float inv = 1.0f / s;
#pragma unroll
    for (int k = 0; k < kEMax; ++k) pr[k] *= inv;
    if (top_p < 1.0f) {
        // smallest value t with mass(p > t) < top_p: bisection on the bit pattern
        // of the (non-negative) threshold; mass_gt is non-increasing in t
        unsigned lo = 0u, hi = 0x3F800000u;             // mass_gt(1.0) = 0 < top_p
        while (lo < hi) {
            const unsigned mid = lo + (hi - lo) / 2;
            const float t = __uint_as_float(mid);
            float m = 0.f;
#pragma unroll
            for (int k = 0; k < kEMax; ++k)
                if (c.lo + k < c.hi) m += pr[k] > t ? pr[k] : 0.f;
            m = block_sum(m, c.red);
            if (m < top_p)
                hi = mid;
            else
                lo = mid + 1;
        }
        // lo: smallest threshold whose strictly-greater mass is below top_p; the
        // boundary value is the largest p_v <= that threshold that still fits
        const float t = __uint_as_float(lo);
        float cand = -1.f;
#pragma unroll
        for (int k = 0; k < kEMax; ++k)
            if (c.lo + k < c.hi && pr[k] <= t) cand = fmaxf(cand, pr[k]);
        const float b = block_max(cand, c.red);         // boundary value (ties possible)
        float above = 0.f;
        int nt = 0;
#pragma unroll
        for (int k = 0; k < kEMax; ++k) {
            if (c.lo + k >= c.hi) continue;
            above += pr[k] > b ? pr[k] : 0.f;
            nt += pr[k] == b ? 1 : 0;
        }
        above = block_sum(above, c.red);
        // tokens equal to b keep their id order: exclusive prefix count per thread
        __syncthreads();
        int* cnt = (int*)c.red.i;                       // reuse: [32] per-wave partial sums
        int incl = nt;
        const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
        for (int o = 1; o < 64; o <<= 1) {
            const int y = __shfl_up(incl, o);
            if (lane >= o) incl += y;
        }
        if (lane == 63) cnt[w] = incl;
        __syncthreads();
        int before = incl - nt;
        for (int k = 0; k < w; ++k) before += cnt[k];
        __syncthreads();
        float kept = 0.f;
        int j = before;
#pragma unroll
        for (int k = 0; k < kEMax; ++k) {
            if (c.lo + k >= c.hi) continue;
            bool keep = pr[k] > b;
            if (pr[k] == b && b > 0.f) {
                keep = above + (float)j * b < top_p;
                ++j;
            }
            if (!keep) pr[k] = 0.f;
            kept += pr[k];
        }
        kept = block_sum(kept, c.red);
        const float ik = 1.0f / kept;
#pragma unroll
        for (int k = 0; k < kEMax; ++k) pr[k] *= ik;
    }
    if (vec4(c)) {
#pragma unroll
        for (int k = 0; k < kEMax; k += 4)
            if (c.lo + k < c.hi) st4(p, c.lo + k, make_float4(pr[k], pr[k + 1], pr[k + 2], pr[k + 3]));
    } else {
#pragma unroll
        for (int k = 0; k < kEMax; ++k)
            if (c.lo + k < c.hi) p[c.lo + k] = pr[k];
    }
}

// exponential race over weights w >= 0 (w_v = 0 never wins)
__device__ int race(const Ctx& c, const float* w, unsigned long long seed, int seq, int pos, int ev) {
    float bv = -INFINITY;
    int bi = -1;
    const bool v4 = vec4(c);
    for (int v0 = c.lo & ~3; v0 < c.hi; v0 += 4) {
        const P4 r = philox((unsigned long long)(v0 >> 2), (unsigned long long)pos, (unsigned long long)ev, 0ull,
                            seed, (unsigned long long)seq);
        float4 w4 = make_float4(0.f, 0.f, 0.f, 0.f);
        if (v4) w4 = ld4(w, v0);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int v = v0 + e;
            if (v < c.lo || v >= c.hi) continue;
            const float wv = v4 ? get4(w4, e) : w[v];
            if (!(wv > 0.f)) continue;
            const float sc = wv / -logf(u23_open(r.x[e]));
            if (beats(sc, v, bv, bi)) {
                bv = sc;
                bi = v;
            }
        }
    }
    return block_argmax(bv, bi, c.red);
}

// q[x] = 0 and the rest renormalised; returns false when no mass is left
__device__ bool mask_renorm(const Ctx& c, float* q, int x) {
    if (x >= c.lo && x < c.hi) q[x] = 0.f;
    float s = 0.f;
    if (vec4(c)) {
        for (int v = c.lo; v < c.hi; v += 4) {
            const float4 a = ld4(q, v);
            s += a.x;
            s += a.y;
            s += a.z;
            s += a.w;
        }
    } else {
        for (int v = c.lo; v < c.hi; ++v) s += q[v];
    }
    s = block_sum(s, c.red);
    if (!(s > 0.f)) return false;
    const float inv = 1.0f / s;
    if (vec4(c)) {
        for (int v = c.lo; v < c.hi; v += 4) {
            float4 a = ld4(q, v);
            a.x *= inv;
            a.y *= inv;
            a.z *= inv;
            a.w *= inv;
            st4(q, v, a);
        }
    } else {
        for (int v = c.lo; v < c.hi; ++v) q[v] *= inv;
    }
    __syncthreads();
    return true;
}

// out = mu (-) nu; returns false (and copies mu) when there is no positive mass
__device__ bool residual(const Ctx& c, const float* mu, const float* nu, float* out) {
    float s = 0.f;
    const bool v4 = vec4(c);
    if (v4) {
        for (int v = c.lo; v < c.hi; v += 4) {
            const float4 a = ld4(mu, v), b = ld4(nu, v);
            float4 d;
            d.x = fmaxf(a.x - b.x, 0.f);
            d.y = fmaxf(a.y - b.y, 0.f);
            d.z = fmaxf(a.z - b.z, 0.f);
            d.w = fmaxf(a.w - b.w, 0.f);
            st4(out, v, d);
            s += d.x;
            s += d.y;
            s += d.z;
            s += d.w;
        }
    } else {
        for (int v = c.lo; v < c.hi; ++v) {
            const float d = fmaxf(mu[v] - nu[v], 0.f);
            out[v] = d;
            s += d;
        }
    }
    s = block_sum(s, c.red);
    if (!(s > 0.f)) {
        if (v4)
            for (int v = c.lo; v < c.hi; v += 4) st4(out, v, ld4(mu, v));
        else
            for (int v = c.lo; v < c.hi; ++v) out[v] = mu[v];
        __syncthreads();
        return false;
    }
    const float inv = 1.0f / s;
    if (v4) {
        for (int v = c.lo; v < c.hi; v += 4) {
            float4 a = ld4(out, v);
            a.x *= inv;
            a.y *= inv;
            a.z *= inv;
            a.w *= inv;
            st4(out, v, a);
        }
    } else {
        for (int v = c.lo; v < c.hi; ++v) out[v] *= inv;
    }
    __syncthreads();
    return true;
}

// out = in over the thread's ids
__device__ void copy_row(const Ctx& c, const float* in, float* out) {
    if (vec4(c))
        for (int v = c.lo; v < c.hi; v += 4) st4(out, v, ld4(in, v));
    else
        for (int v = c.lo; v < c.hi; ++v) out[v] = in[v];
}

__device__ float accept_u(unsigned long long seed, int seq, int pos, int ev) {
    return u24(philox(0ull, (unsigned long long)pos, (unsigned long long)ev, 0ull, seed, (unsigned long long)seq).x[0]);
}

__global__ void __launch_bounds__(kThreads) k_finalize_sample(Sched s, int fin_op, const float* logits) {
    const int i = blockIdx.x;
    if (i >= *s.nC) return;
    __shared__ float rf[32];
    __shared__ int ri[32];
    __shared__ float sh[4];
    const int V = s.g.V;
    Ctx c;
    c.V = V;
    c.E = (V + blockDim.x - 1) / blockDim.x;
    c.lo = min(V, (int)threadIdx.x * c.E);
    c.hi = min(V, c.lo + c.E);
    c.red = Red{rf, ri};
    const Row row = s.rowsC[i];
    const int b = row.slot, seq = row.seq, pd = row.pos + 1;     // position being decided
    const unsigned long long seed = *s.seed;
    float* p = s.work + (size_t)i * V;
    readout_dist(c, logits + (size_t)i * V, p, s.temperature, s.top_p);
    __syncthreads();
    const int mode = *s.mode;
    int tok = -1, aux = 0;
    if (fin_op == FIN_TARGET || mode == MODE_VANILLA || mode == MODE_FORCED) {
        if (fin_op == FIN_TARGET || row.depth == s.R) tok = race(c, p, seed, seq, pd, EV_TARGET);
    } else if (row.depth == s.d1) {
        float* q1 = s.q1 + (size_t)b * V;
        copy_row(c, p, q1);
        tok = race(c, p, seed, seq, pd, EV_DRAFT1);
    } else if (s.d2 > 0 && row.depth == s.d2) {
        const float* q1 = s.q1 + (size_t)b * V;
        const int x1 = s.s_x1[b];
        float* q2 = s.q2 + (size_t)b * V;
        bool open;
        if (x1 < 0 || x1 >= V) {                       // no first draft recorded: no second proposal
            open = false;
        } else if (s.variant == 0) {
            open = p[x1] < q1[x1];
            if (open && !residual(c, p, q1, q2) && threadIdx.x == 0)
                atomicAdd((unsigned long long*)&s.stats[ST_ZERO_MASS], 1ull);
        } else {
            if (s.variant == 1) {
                if (!residual(c, p, q1, q2) && threadIdx.x == 0)
                    atomicAdd((unsigned long long*)&s.stats[ST_ZERO_MASS], 1ull);
            } else {
                copy_row(c, p, q2);
                __syncthreads();
            }
            open = mask_renorm(c, q2, x1);
        }
        if (open) tok = race(c, q2, seed, seq, pd, EV_DRAFT2);
        aux = open ? 1 : 0;
    } else if (row.depth == s.R) {
        const float* q1 = s.q1 + (size_t)b * V;
        const int x1 = s.s_x1[b];
        const bool drafted = x1 >= 0 && x1 < V;         // the same in every thread of the workgroup
        if (threadIdx.x == 0) {
            const float u = accept_u(seed, seq, pd, EV_ACC1);
            sh[0] = drafted && u < fminf(1.0f, p[x1] / q1[x1]) ? 1.f : 0.f;
        }
        __syncthreads();
        if (!drafted) {                                 // nothing to verify: draw the token from p
            tok = race(c, p, seed, seq, pd, EV_RESAMPLE);
            aux = 0;
        } else if (sh[0] != 0.f) {
            tok = x1;
            aux = 1;
        } else {
            // rho1 = p (-) q1, written over p's buffer through a second pass
            float* rho = p;
            float* tmp = s.q1 + (size_t)b * V;          // q1 is dead after this point: reuse as scratch
            if (!residual(c, p, q1, tmp) && threadIdx.x == 0)
                atomicAdd((unsigned long long*)&s.stats[ST_ZERO_MASS], 1ull);
            copy_row(c, tmp, rho);
            __syncthreads();
            bool done = false;
            if (s.s_gate[b]) {
                const float* q2 = s.q2 + (size_t)b * V;
                const int x2 = s.s_x2[b];
                if (threadIdx.x == 0) {
                    const float u = accept_u(seed, seq, pd, EV_ACC2);
                    sh[1] = u < fminf(1.0f, rho[x2] / q2[x2]) ? 1.f : 0.f;
                }
                __syncthreads();
                if (sh[1] != 0.f) {
                    tok = x2;
                    aux = 2;
                    done = true;
                } else {
                    if (!residual(c, rho, q2, tmp) && threadIdx.x == 0)
                        atomicAdd((unsigned long long*)&s.stats[ST_ZERO_MASS], 1ull);
                    copy_row(c, tmp, rho);
                    __syncthreads();
                }
            }
            if (!done) {
                tok = race(c, rho, seed, seq, pd, EV_RESAMPLE);
                aux = 0;
            }
        }
    }
    if (threadIdx.x == 0) {
        s.ro_tok[i] = tok;
        s.ro_aux[i] = aux;
    }
}

hipError_t launch_finalize_sample(const Sched& s, int fin_op, const float* logits, int rows_cap, hipStream_t st) {
    hipLaunchKernelGGL(k_finalize_sample, dim3(rows_cap), dim3(kThreads), 0, st, s, fin_op, logits);
    return hipGetLastError();
}

}  // namespace ls
