// Decode attention over per-depth KV caches.
//
// Computation at recurrent depth r needs the keys/values of the same depth
// (implementation details, KV cache management): a row at depth r and block
// layer l attends over positions 0..pos with the (r, l) cache.  Positions below
// the sequence's committed length come from the committed cache; positions of
// the row's in-flight ancestors come from their branch slots (a child reuses
// its parent's prefix instead of copying it); the row's own position comes from
// its own slot, written by the QKV epilogue of the same layer.
//
// One workgroup per (head, row).  Its wavefronts take kChunk-position chunks of
// the *logical* positions before the row's own, and the own position as one
// more partial; inside a chunk a position's head slice spans a few lanes (one
// 16-byte load each), every key and value load of the chunk is issued before
// any is used, and a score reduces over its position's lanes.  Partials (o,
// max, sum) stay in LDS and are combined in chunk order, so a row's result
// depends only on the values it reads, never on where they are stored or how
// many rows run: vanilla decoding and LoopSpec get bit-identical outputs.
#include "ls_attn_dev.h"

namespace ls {

// DH: head dim; one workgroup per (head, row).
template <typename WT, int DH>
__global__ void __launch_bounds__(512) k_attn(AttnParams p) {
    extern __shared__ float smem[];
    const int m = blockIdx.y;
    if (m >= *p.nrows) return;
    attn_item<WT, DH, false>(p, m, blockIdx.x, smem);
}

// Shared-prefix task attention for decode row lists (KV cache management of
// the pipelined decode: the rows of one sequence at one depth read the same
// committed keys and values).  Rows with the same (sequence, depth, committed
// length) form a group led by its lowest row index.  The work is a list of
// one-wave tasks spread over the whole grid, per head: every chunk of 64
// positions wholly below the committed length once per group (its keys and
// values loaded once and scored against each member's query), then per row
// the chunks that hold its in-flight ancestors and its own position.  Each
// task stores its partial (o, max, sum) per member at device scope and counts
// it on the member's (row, head) counter; the task that completes a (row,
// head) combines its partials in chunk order, writes the output and resets
// the counter for the next launch.  A row's partials and their combination
// are the same arithmetic whatever group it falls in, so grouped rows equal
// rows computed alone bit for bit.
template <typename WT, int DH>
__device__ __forceinline__ void store_partial(float* dst, const float (&acc)[KV<WT>::E], float mx, float l) {
    using A = AttnGeo<WT, DH>;
    constexpr int E = A::E;
    const int lane = tid_local() & 63, d8 = lane % A::LPP, grp = lane / A::LPP;
    if (grp == 0 && d8 < A::NK) {
#pragma unroll
        for (int e = 0; e < E; ++e) st_f32<true>(dst + d8 * E + e, acc[e]);
    }
    if (lane == 0) {
        st_f32<true>(dst + DH, mx);
        st_f32<true>(dst + DH + 1, l);
    }
}

// The output of (row m, head) from its n partials at base ([n][DH + 2], device
// scope): maximum over the chunk maxima, then the chunk values and weight sums
// weighted by exp2(max_c - max) and summed in chunk order.
template <typename WT, int DH>
__device__ __forceinline__ void combine_partials(const AttnParams& p, int m, int head, int n, const float* base) {
    constexpr int DPL = (DH + 63) / 64, CB = 16;
    const int lane = tid_local() & 63;
    float gmx = -INFINITY;
    for (int c0 = 0; c0 < n; c0 += 64)
        if (c0 + lane < n) gmx = fmaxf(gmx, ld_f32<true>(base + (size_t)(c0 + lane) * (DH + 2) + DH));
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) gmx = fmaxf(gmx, __shfl_xor(gmx, o));
    float lsum = 0.f, o[DPL];
#pragma unroll
    for (int j = 0; j < DPL; ++j) o[j] = 0.f;
    for (int c0 = 0; c0 < n; c0 += 64) {
        const int cl = c0 + lane;
        const float mc = cl < n ? ld_f32<true>(base + (size_t)cl * (DH + 2) + DH) : -INFINITY;
        const float lc = cl < n ? ld_f32<true>(base + (size_t)cl * (DH + 2) + DH + 1) : 0.f;
        const float wc = cl < n ? exp2_fast(mc - gmx) : 0.f;
        const int nb = n - c0 < 64 ? n - c0 : 64;
        for (int i0 = 0; i0 < nb; i0 += CB) {
            float v[CB][DPL];
#pragma unroll
            for (int i = 0; i < CB; ++i)
#pragma unroll
                for (int j = 0; j < DPL; ++j) {
                    const int d = lane + 64 * j;
                    v[i][j] = (i0 + i < nb && d < DH) ? ld_f32<true>(base + (size_t)(c0 + i0 + i) * (DH + 2) + d)
                                                      : 0.f;
                }
#pragma unroll
            for (int i = 0; i < CB; ++i) {
                if (i0 + i >= nb) break;
                const float w = lane_read(wc, i0 + i), lcc = lane_read(lc, i0 + i);
                lsum = fmaf(lcc, w, lsum);
#pragma unroll
                for (int j = 0; j < DPL; ++j) o[j] = fmaf(v[i][j], w, o[j]);
            }
        }
    }
#pragma unroll
    for (int j = 0; j < DPL; ++j) {
        const int d = lane + 64 * j;
        if (d >= DH) break;
        const float r = o[j] / lsum;
        const size_t idx = (size_t)m * p.g.h + head * DH + d;
        if (sizeof(WT) == 2)
            ((uint16_t*)p.out)[idx] = f2h(r);
        else
            ((float*)p.out)[idx] = r;
    }
}

// Count `add` stored partials of (row m, head); the task completing its n
// partials combines them and clears the counter.
template <typename WT, int DH>
__device__ __forceinline__ void count_partials(const AttnParams& p, int m, int head, int n, int add,
                                               const float* base, unsigned* cnt) {
    const int lane = tid_local() & 63;
    unsigned old = 0;
    if (lane == 0)
        old = __hip_atomic_fetch_add(cnt + m * p.g.H + head, (unsigned)add, __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT);
    old = __shfl(old, 0);
    if (old + add != (unsigned)n) return;
    combine_partials<WT, DH>(p, m, head, n, base);
    if (lane == 0) __hip_atomic_store(cnt + m * p.g.H + head, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// A row's units are the chunks before its own position (units 0 .. np - 1,
// the first ns of them wholly committed and shared by its group) and its own
// position (unit np).  A task covers tu consecutive units of one head, of the
// group's shared units or of the row's own ones, tu = task_units(ns): a
// function of the committed length only, so every member of a group -- and
// the same row alone -- cuts its units the same way.  The task merges its
// units' partials in unit order into one partial per row.
__device__ __forceinline__ int task_units(int ns) {
    const int u = ns / 16;
    return u < 1 ? 1 : u > 8 ? 8 : u;
}

template <int E>
__device__ __forceinline__ void merge_partial(float (&acc_r)[E], float& m_r, float& l_r, const float (&acc)[E], float m,
                                              float l) {
    const float mn = fmaxf(m_r, m);
    const float so = exp2_fast(m_r - mn), sn = exp2_fast(m - mn);
#pragma unroll
    for (int e = 0; e < E; ++e) acc_r[e] = fmaf(acc_r[e], so, acc[e] * sn);
    l_r = fmaf(l_r, so, l * sn);
    m_r = mn;
}

constexpr int kGroupBatch = 2;      // members of a group one shared task carries at a time

template <typename WT, int DH>
__global__ void __launch_bounds__(256) k_attn_tasks(AttnParams p, float* part, unsigned* cnt) {
    using A = AttnGeo<WT, DH>;
    constexpr int E = A::E, NIT = A::NIT, GB = kGroupBatch;
    const int M = *p.nrows;
    if (M <= 0) return;
    const int tid = tid_local(), wave = tid >> 6, lane = tid & 63;
    const int H = p.g.H, cap = p.chunks_cap;
    // lane i < M describes row i: its group (same sequence, depth and
    // committed length) and its task count per head
    int seq = -1, depth = -1, tdone = -1, pos = 0;
    if (lane < M) {
        seq = p.rows[lane].seq;
        depth = p.rows[lane].depth;
        tdone = p.rows[lane].tdone;
        pos = p.rows[lane].pos;
    }
    unsigned long long gmask = 0;
    for (int i = 0; i < M; ++i) {
        const int si = __shfl(seq, i), di = __shfl(depth, i), ti = __shfl(tdone, i);
        const unsigned long long mk = __ballot(lane < M && seq == si && depth == di && tdone == ti);
        if (lane == i) gmask = mk;
    }
    const bool leader = lane < M && (int)__builtin_ctzll(gmask) == lane;
    const int ns = lane < M ? tdone / kChunk : 0;                 // units the group shares
    const int np = lane < M ? (pos + kChunk - 1) / kChunk : 0;    // the own position's unit
    const int tu = task_units(ns);
    const int nsh = (ns + tu - 1) / tu;                           // shared tasks (partials) of the group
    const int nrow = nsh + (np - ns + 1 + tu - 1) / tu;           // partials of the row
    const int tl = lane < M ? (leader ? nrow : nrow - nsh) : 0;   // tasks this row leads, per head
    int pre = tl * H;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int v = __shfl_up(pre, o);
        if (lane >= o) pre += v;
    }
    const int total = __shfl(pre, 63);
    const size_t per = (size_t)(cap + 1) * (DH + 2);
    const int d8 = lane % A::LPP;
    for (int k = blockIdx.x * 4 + wave; k < total; k += gridDim.x * 4) {
        const int m = __popcll(__ballot(lane < M && pre <= k));
        const int before = m ? __shfl(pre, m - 1) : 0;
        const int tm = __shfl(tl, m), r = k - before, head = r / tm, cc = r - head * tm;
        const bool lead = __shfl((int)leader, m) != 0;
        const int nshm = __shfl(nsh, m), nsm = __shfl(ns, m), npm = __shfl(np, m), tum = __shfl(tu, m);
        const int nrm = __shfl(nrow, m);
        const int t = kv_table(p.g, p.stack, p.layer, __shfl(depth, m));
        if (lead && cc < nshm) {
            // shared units: each chunk's keys and values loaded once per batch
            // of members, a merged partial per member
            unsigned long long left = ((unsigned long long)(unsigned)__shfl((int)(gmask >> 32), m) << 32) |
                                      (unsigned)__shfl((int)gmask, m);
            const unsigned long long mem = left;
            const int u0 = cc * tum, u1 = u0 + tum < nsm ? u0 + tum : nsm;
            while (left) {
                int jb[GB];
#pragma unroll
                for (int b = 0; b < GB; ++b) {
                    jb[b] = -1;
                    if (left) {
                        jb[b] = __builtin_ctzll(left);
                        left &= left - 1;
                    }
                }
                float accs[GB][E], ms[GB], ls[GB];
#pragma nounroll
                for (int c = u0; c < u1; ++c) {
                    const int cu = __builtin_amdgcn_readfirstlane(c), p0 = cu * kChunk;
                    u32x4 kr[NIT], vr[NIT];
                    chunk_kv_committed<WT, DH>(p, __builtin_amdgcn_readfirstlane(__shfl(seq, m)),
                                               __builtin_amdgcn_readfirstlane(t),
                                               __builtin_amdgcn_readfirstlane(head), p0, kr, vr);
#pragma unroll
                    for (int b = 0; b < GB; ++b) {
                        if (jb[b] < 0) continue;
                        const int j = jb[b];
                        const int plast = __builtin_amdgcn_readfirstlane(__shfl(pos, j) - 1);
                        const float* qsrc = p.q + (size_t)j * p.g.h + head * DH + d8 * E;
                        u32x4 qr[E / 4];
#pragma unroll
                        for (int e = 0; e < E / 4; ++e)
                            qr[e] = d8 < A::NK ? *(const u32x4*)(qsrc + 4 * e) : u32x4{0u, 0u, 0u, 0u};
                        float acc[E], mx, l;
                        chunk_math<WT, DH>(p, qr, kr, vr, p0, plast, acc, mx, l);
                        if (c == u0) {
#pragma unroll
                            for (int e = 0; e < E; ++e) accs[b][e] = acc[e];
                            ms[b] = mx;
                            ls[b] = l;
                        } else {
                            merge_partial<E>(accs[b], ms[b], ls[b], acc, mx, l);
                        }
                    }
                }
#pragma unroll
                for (int b = 0; b < GB; ++b)
                    if (jb[b] >= 0)
                        store_partial<WT, DH>(part + (size_t)(jb[b] * H + head) * per + (size_t)cc * (DH + 2),
                                              accs[b], ms[b], ls[b]);
            }
            __builtin_amdgcn_s_waitcnt(0);              // the partials are visible device-wide
            for (unsigned long long x = mem; x; x &= x - 1) {
                const int j = __builtin_ctzll(x);
                const int npj = (__shfl(pos, j) + kChunk - 1) / kChunk;
                const int nj = nshm + (npj - nsm + 1 + tum - 1) / tum;
                count_partials<WT, DH>(p, j, head, nj, 1, part + (size_t)(j * H + head) * per, cnt);
            }
            continue;
        }
        // the row's own units: chunks holding its in-flight ancestors, then its own position
        const int b = cc - (lead ? nshm : 0);            // own task index
        const int u0 = nsm + b * tum, u1 = u0 + tum < npm + 1 ? u0 + tum : npm + 1;
        const Row row = row_head(p.rows, m);
        float* base = part + (size_t)(m * H + head) * per;
        float acc_r[E], m_r = -INFINITY, l_r = 0.f;
#pragma nounroll
        for (int c = u0; c < u1; ++c) {
            float acc[E], mx, l;
            if (c < npm)
                attn_chunk<WT, DH, false>(p, row, m, p.rows[m].anc, t, head, c, row.pos - 1, acc, mx, l);
            else
                attn_own<WT, DH, false>(p, row, m, p.rows[m].anc, t, head, acc, mx, l);
            if (c == u0) {
#pragma unroll
                for (int e = 0; e < E; ++e) acc_r[e] = acc[e];
                m_r = mx;
                l_r = l;
            } else {
                merge_partial<E>(acc_r, m_r, l_r, acc, mx, l);
            }
        }
        store_partial<WT, DH>(base + (size_t)(nshm + b) * (DH + 2), acc_r, m_r, l_r);
        __builtin_amdgcn_s_waitcnt(0);
        count_partials<WT, DH>(p, m, head, nrm, 1, base, cnt);
    }
}

int attention_waves(int chunks_cap) { return chunks_cap < 8 ? chunks_cap : 8; }


// partials of every chunk and of the own position, and one weight per partial
size_t attention_lds_bytes(int chunks_cap, int dh) { return (size_t)(chunks_cap + 1) * (dh + 3) * 4; }

size_t attention_partials_floats(int rows, int heads, int chunks_cap, int dh) {
    return (size_t)rows * heads * (chunks_cap + 1) * (dh + 2);
}

// grid of the task attention: four one-wave tasks per workgroup, four workgroups per CU
static int task_grid() {
    static int g = 0;
    if (!g) {
        int dev = 0, cus = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
            cus = 256;
        g = cus * 4;
    }
    return g;
}

template <typename WT, int DH>
static void launch_dh(const AttnParams& p, int m_cap, float* part, unsigned* cnt, hipStream_t st) {
    AttnParams q = p;
    if (part) {
        void* args[] = {(void*)&q, (void*)&part, (void*)&cnt};
        (void)ls_launch((const void*)k_attn_tasks<WT, DH>, dim3(task_grid()), dim3(256), args, 0, st);
        return;
    }
    const int w = attention_waves(p.chunks_cap);
    void* args[] = {(void*)&q};
    (void)ls_launch((const void*)k_attn<WT, DH>, dim3(p.g.H, m_cap), dim3(64 * w),
                    args, attention_lds_bytes(p.chunks_cap, DH), st);
}

// head dims: a head slice is at most 16 lanes of 16 bytes (fp32: dh <= 64)
template <typename WT>
static hipError_t launch_t(const AttnParams& p, int m_cap, float* part, unsigned* cnt, hipStream_t st) {
    switch (p.g.dh) {
        case 16: launch_dh<WT, 16>(p, m_cap, part, cnt, st); break;
        case 32: launch_dh<WT, 32>(p, m_cap, part, cnt, st); break;
        case 64: launch_dh<WT, 64>(p, m_cap, part, cnt, st); break;
        default:
            if constexpr (sizeof(WT) == 2) {
                if (p.g.dh == 96) {
                    launch_dh<WT, 96>(p, m_cap, part, cnt, st);
                    break;
                }
                if (p.g.dh == 128) {
                    launch_dh<WT, 128>(p, m_cap, part, cnt, st);
                    break;
                }
            }
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <typename WT>
static hipError_t allow(int bytes) {
    const void* f[] = {(const void*)k_attn<WT, 16>, (const void*)k_attn<WT, 32>, (const void*)k_attn<WT, 64>};
    for (const void* x : f) {
        hipError_t e = hipFuncSetAttribute(x, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
        if (e != hipSuccess) return e;
    }
    if constexpr (sizeof(WT) == 2) {
        const void* g[] = {(const void*)k_attn<WT, 96>, (const void*)k_attn<WT, 128>};
        for (const void* x : g) {
            hipError_t e = hipFuncSetAttribute(x, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
            if (e != hipSuccess) return e;
        }
    }
    return hipSuccess;
}

hipError_t attention_prepare(int lds_bytes) {
    hipError_t e = allow<uint16_t>(lds_bytes);
    return e != hipSuccess ? e : allow<float>(lds_bytes);
}

hipError_t launch_attention(const AttnParams& p, bool bf16, int m_cap, float* part, unsigned* cnt, hipStream_t st) {
    return bf16 ? launch_t<uint16_t>(p, m_cap, part, cnt, st) : launch_t<float>(p, m_cap, part, cnt, st);
}

}  // namespace ls
