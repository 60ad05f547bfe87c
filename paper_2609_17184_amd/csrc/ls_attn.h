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
// fp32 words of the shared-prefix task attention's partials ([rows][heads][chunks_cap + 1][dh + 2])
size_t attention_partials_floats(int rows, int heads, int chunks_cap, int dh);
int attention_waves(int chunks_cap);
hipError_t attention_prepare(int lds_bytes);   // allow the dynamic LDS size
// part != NULL: the shared-prefix task attention (part: its partials; cnt:
// [rows][heads] counters, zero between launches); else one workgroup per (head, row)
hipError_t launch_attention(const AttnParams& p, bool bf16, int m_cap, float* part, unsigned* cnt, hipStream_t st);

}  // namespace ls
