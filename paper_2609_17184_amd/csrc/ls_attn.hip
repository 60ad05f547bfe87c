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

int attention_waves(int chunks_cap) { return chunks_cap < 8 ? chunks_cap : 8; }

// partials of every chunk and of the own position, and one weight per partial
size_t attention_lds_bytes(int chunks_cap, int dh) { return (size_t)(chunks_cap + 1) * (dh + 3) * 4; }

template <typename WT, int DH>
static void launch_dh(const AttnParams& p, int m_cap, hipStream_t st) {
    const int w = attention_waves(p.chunks_cap);
    AttnParams q = p;
    void* args[] = {(void*)&q};
    (void)ls_launch((const void*)k_attn<WT, DH>, dim3(p.g.H, m_cap), dim3(64 * w),
                    args, attention_lds_bytes(p.chunks_cap, DH), st);
}

// head dims: a head slice is at most 16 lanes of 16 bytes (fp32: dh <= 64)
template <typename WT>
static hipError_t launch_t(const AttnParams& p, int m_cap, hipStream_t st) {
    switch (p.g.dh) {
        case 16: launch_dh<WT, 16>(p, m_cap, st); break;
        case 32: launch_dh<WT, 32>(p, m_cap, st); break;
        case 64: launch_dh<WT, 64>(p, m_cap, st); break;
        default:
            if constexpr (sizeof(WT) == 2) {
                if (p.g.dh == 96) {
                    launch_dh<WT, 96>(p, m_cap, st);
                    break;
                }
                if (p.g.dh == 128) {
                    launch_dh<WT, 128>(p, m_cap, st);
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

hipError_t launch_attention(const AttnParams& p, bool bf16, int m_cap, hipStream_t st) {
    return bf16 ? launch_t<uint16_t>(p, m_cap, st) : launch_t<float>(p, m_cap, st);
}

}  // namespace ls
