// Achievable HBM read bandwidth of this GPU.  Decoding streams the model's
// weights once per step and is bound by memory bandwidth (the premise of
// Sec. 1 and 3.1), so the bandwidth the decoding kernels reach is read
// against two ceilings: the published peak and what a plain streaming read
// of the same number of bytes reaches here.  The probe reads a buffer with
// the access pattern of the weight-streaming layers: 16-byte non-temporal
// loads, consecutive lanes on consecutive chunks, several loads in flight
// per thread, a grid-stride loop over a chosen number of work-groups.
#include "sd.h"

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <string>

#include "host_api.h"

namespace {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int PROBE_THREADS = 256;

// XOR of everything read; stored only when it equals key, which the caller
// picks so that it (almost) never does: the loads cannot be dropped.
// PROBE_UNROLL loads of 16 bytes are in flight per thread.
template <int PROBE_UNROLL>
__global__ __launch_bounds__(PROBE_THREADS) void k_read_probe(const u32x4_t *p, size_t n16, uint32_t key,
                                                              uint32_t *sink) {
    const size_t stride = (size_t)gridDim.x * PROBE_THREADS;
    size_t i = (size_t)blockIdx.x * PROBE_THREADS + threadIdx.x;
    uint32_t acc = 0;
    for (; i + (PROBE_UNROLL - 1) * stride < n16; i += PROBE_UNROLL * stride) {
        u32x4_t v[PROBE_UNROLL];
#pragma unroll
        for (int u = 0; u < PROBE_UNROLL; ++u)
            v[u] = __builtin_nontemporal_load(p + i + u * stride);
#pragma unroll
        for (int u = 0; u < PROBE_UNROLL; ++u)
            acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
    }
    for (; i < n16; i += stride) {
        const u32x4_t v = __builtin_nontemporal_load(p + i);
        acc ^= v[0] ^ v[1] ^ v[2] ^ v[3];
    }
    if (acc == key)
        sink[0] = acc;
}

}  // namespace

extern "C" sd_status sd_measure_read_bandwidth(const void *buf, size_t bytes, int32_t wg_per_cu,
                                               int32_t loads_in_flight, int32_t iters, void *sink, void *hip_stream,
                                               double *ms_out) {
    if (!buf || !sink || !ms_out || bytes < 16 || (bytes & 15) || ((uintptr_t)buf & 15) || wg_per_cu < 1 ||
        wg_per_cu > 64 || iters < 1 || (loads_in_flight != 2 && loads_in_flight != 4 && loads_in_flight != 8 &&
                                        loads_in_flight != 16))
        return sdk::report(SD_ERR_INVALID_ARG, "read probe: buf and sink must be set, bytes a positive multiple of "
                                               "16 at a 16-byte aligned address, wg_per_cu in [1, 64], "
                                               "loads_in_flight 2, 4, 8 or 16, iters >= 1");
    hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess || (s && hipStreamGetDevice(s, &dev) != hipSuccess) ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        return sdk::report(SD_ERR_DEVICE, "read probe: device query failed");
    hipEvent_t a = nullptr, b = nullptr;
    if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess) {
        if (a)
            (void)hipEventDestroy(a);
        return sdk::report(SD_ERR_DEVICE, "read probe: event creation failed");
    }
    const size_t n16 = bytes / 16;
    const dim3 grid((unsigned)(cus * wg_per_cu)), block(PROBE_THREADS);
    double total = 0.0;
    sd_status st = SD_OK;
    for (int it = 0; it < iters && st == SD_OK; ++it) {
        // the events are attached to the dispatch: they time the kernel's own start and end
        const u32x4_t *p = reinterpret_cast<const u32x4_t *>(buf);
        const uint32_t key = 0x9e3779b9u + (uint32_t)it;
        uint32_t *sk = reinterpret_cast<uint32_t *>(sink);
        if (loads_in_flight == 2)
            hipExtLaunchKernelGGL(k_read_probe<2>, grid, block, 0, s, a, b, 0, p, n16, key, sk);
        else if (loads_in_flight == 4)
            hipExtLaunchKernelGGL(k_read_probe<4>, grid, block, 0, s, a, b, 0, p, n16, key, sk);
        else if (loads_in_flight == 8)
            hipExtLaunchKernelGGL(k_read_probe<8>, grid, block, 0, s, a, b, 0, p, n16, key, sk);
        else
            hipExtLaunchKernelGGL(k_read_probe<16>, grid, block, 0, s, a, b, 0, p, n16, key, sk);
        float ms = 0.0f;
        if (hipGetLastError() != hipSuccess || hipEventSynchronize(b) != hipSuccess ||
            hipEventElapsedTime(&ms, a, b) != hipSuccess)
            st = sdk::report(SD_ERR_DEVICE, "read probe: launch or timing failed");
        total += ms;
    }
    (void)hipEventDestroy(a);
    (void)hipEventDestroy(b);
    if (st == SD_OK)
        *ms_out = total / iters;
    return st;
}
