// Launch interface of the per-depth decode attention (ls_attn.hip).
#pragma once
#include "ls_common.h"

namespace ls {

struct AttnParams {
    Geo g;
    const int32_t* nrows;
    const Row* rows;
    const float* q;            // [M][h] rotated queries
    const void* kvc;           // committed cache [seq][T][2][H][max_ctx][dh]
    const void* kvs;           // slot cache [slot][T][2][h]
    int stack, layer;
    int chunks_cap;            // ceil(max_ctx / 64)
    void* out;                 // [M][h] attention output (weight dtype)
    int32_t* err;              // persistent pass: kErrPoll when a read gave up waiting
};

size_t attention_lds_bytes(int chunks_cap, int dh);
int attention_waves(int chunks_cap);
hipError_t attention_prepare(int lds_bytes);   // allow the dynamic LDS size
hipError_t launch_attention(const AttnParams& p, bool bf16, int m_cap, hipStream_t st);

}  // namespace ls
