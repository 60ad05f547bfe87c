// Vocabulary-sharded sampling readout (ls_sample.hip): layout of the per-row
// synchronisation scratch and the launchers the runtime uses.
#pragma once
#include "ls_sched.h"

namespace ls {

// One readout row is split over NS workgroups ("shards") of kSThreads
// threads; thread t of shard s owns the E consecutive ids starting at
// s * 256 * E + t * E.
constexpr int kSThreads = 256;
constexpr int kSEMax = 16;           // ids per thread
constexpr int kSShardsMax = 16;      // shards per row
static_assert(kSThreads * kSEMax * kSShardsMax >= kSampleMaxVocab, "shards must cover the vocabulary");

struct SGeo {
    int V, E, chunk, NS;
};
// E: the fewest ids per thread (a multiple of 4, at least 4) that cover V
// with at most kSShardsMax shards
__host__ __device__ inline SGeo sample_geo(int V) {
    SGeo g;
    g.V = V;
    int e = (V + kSThreads * kSShardsMax - 1) / (kSThreads * kSShardsMax);
    e = (e + 3) & ~3;
    g.E = e < 4 ? 4 : e;
    g.chunk = kSThreads * g.E;
    g.NS = (V + g.chunk - 1) / g.chunk;
    return g;
}

// Radix selection of the top-p boundary over the bit pattern of the fp32
// probabilities (31 bits below the sign): three rounds of 11, 10 and 10 bits.
constexpr int kRadixBits[3] = {11, 10, 10};
constexpr int kRadixShift[3] = {20, 10, 0};
constexpr int kHistWords = (1 << 11) + (1 << 10) + (1 << 10);

// Per-row scratch of a row split over several shards, in 64-bit words:
//   [kRowCnt]            barrier counter (arrivals of the row's shards)
//   [kRowPart ...)       two banks x kSShardsMax shards x kPartSlots values
//                        published by each shard before a barrier
//   [kRowHist ...)       the three rounds' histograms (count << 44 | mass)
// Zero between launches: the last shard of a row to leave resets it.
constexpr int kPartSlots = 8;
constexpr int kRowCnt = 0;
constexpr int kRowPart = 8;
constexpr int kRowHist = kRowPart + 2 * kSShardsMax * kPartSlots;
constexpr int kRowWords = kRowHist + kHistWords;

// Rows one launch of the standalone cascade handles when a row takes several
// shards (so that every shard of every row in flight is resident at once).
constexpr int kCascadeRowsPerLaunch = 64;

// decode steps: the sampled readout of every C row (Alg. 1 proposals and
// verification); s.srow holds kRowWords words per row
hipError_t launch_finalize_sample(const Sched& s, int fin_op, const float* logits, int rows_cap, hipStream_t st);
// rows whose shards all fit on the GPU at once (0 if unknown)
int sample_rows_resident(int V);
// zero n words of per-row scratch (a fill kernel: safe inside graph capture)
hipError_t launch_zero_words(unsigned long long* p, size_t n, hipStream_t st);

}  // namespace ls
