// Read-stream probe: the HBM read rate a plain streaming kernel reaches, the
// practical ceiling for the weight stream of a decode pass (a measurement aid
// beside the method, used to put the pass's achieved bandwidth in context).
//
// 256 workgroups of 256 threads walk the buffer in grid-stride order, eight
// 16-byte nontemporal loads in flight per thread, every 16-byte vector read
// exactly once per pass; each thread XORs the words it read, so the XOR of
// the per-thread results equals the XOR of the whole buffer (a check that the
// pass covered it).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/loopspec.h"

namespace ls {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
constexpr int kProbeGrid = 256, kProbeThreads = 256, kProbeUnroll = 8;

__global__ void __launch_bounds__(kProbeThreads) k_read_stream(const u32x4_t* __restrict__ p, size_t n,
                                                               uint32_t* out) {
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    uint32_t acc = 0;
    // whole rounds: the last of the kProbeUnroll vectors is below n
    for (; i + (kProbeUnroll - 1) * stride < n; i += kProbeUnroll * stride) {
        u32x4_t v[kProbeUnroll];
#pragma unroll
        for (int u = 0; u < kProbeUnroll; ++u) v[u] = __builtin_nontemporal_load(p + i + u * stride);
#pragma unroll
        for (int u = 0; u < kProbeUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    for (; i < n; i += stride) {
        const u32x4_t v = p[i];
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = acc;
}

}  // namespace ls

extern "C" int loopspec_read_bandwidth(const void* buf, uint64_t bytes, int32_t reps, void* stream,
                                       uint32_t* xor_out, float* gbps) {
    if (!buf || !xor_out || !gbps || reps < 1 || bytes == 0 || bytes % 16 || bytes >= ((uint64_t)1 << 36))
        return LOOPSPEC_EINVAL;
    hipStream_t st = (hipStream_t)stream;
    const size_t n = bytes / 16;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    int rc = LOOPSPEC_OK;
    float ms = 0.f;
    if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) {
        rc = LOOPSPEC_EHIP;
    } else {
        hipLaunchKernelGGL(ls::k_read_stream, dim3(ls::kProbeGrid), dim3(ls::kProbeThreads), 0, st,
                           (const ls::u32x4_t*)buf, n, xor_out);   // untimed first pass
        (void)hipEventRecord(e0, st);
        for (int r = 0; r < reps; ++r)
            hipLaunchKernelGGL(ls::k_read_stream, dim3(ls::kProbeGrid), dim3(ls::kProbeThreads), 0, st,
                               (const ls::u32x4_t*)buf, n, xor_out);
        (void)hipEventRecord(e1, st);
        if (hipGetLastError() != hipSuccess || hipEventSynchronize(e1) != hipSuccess ||
            hipEventElapsedTime(&ms, e0, e1) != hipSuccess || !(ms > 0.f))
            rc = LOOPSPEC_EHIP;
        else
            *gbps = (float)((double)bytes * reps / (ms * 1e-3) / 1e9);
    }
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    return rc;
}
