// Read-bandwidth probe of the device (a measurement tool for the benchmark, not part of
// the verification library): the achievable HBM read rate that the row kernel's
// algorithmic bandwidth is compared with.
//
//   int resispec_probe_read(const void* src, int64_t nbytes, int32_t chunk_bytes,
//                           int32_t policy, int32_t passes, void* sink, hipStream_t stream);
//
// src: device buffer of nbytes bytes, read only.  Each 512-thread workgroup streams one
// contiguous chunk of chunk_bytes bytes with 16-byte buffer loads, four in flight per
// thread, like the row kernel streams one row.  policy 0: ordinary loads; 1: nontemporal
// loads.  passes 1: one read; 2: the chunk is read, then read again in reverse order
// with nontemporal loads (the pattern of a pass followed by a rejection pass over the
// same row).  sink: device buffer of at least nbytes / chunk_bytes uint32 values that
// the kernel writes only if a checksum takes one impossible value (it keeps the loads).
// Returns 0 when launched; 1 for invalid arguments (nothing launched: nbytes and
// chunk_bytes must be positive, chunk_bytes a multiple of 32 KiB and a divisor of
// nbytes, the chunk count below 2^31, policy and passes as above, pointers non-null);
// 2 when the launch fails.  Asynchronous on `stream`.
#include <hip/hip_runtime.h>
#include <cstdint>

namespace {

constexpr int kProbeBlock = 512;
constexpr int kProbeUnroll = 4;
constexpr int kChunkQuantum = kProbeBlock * kProbeUnroll * 16;   // 32 KiB

typedef int v4i __attribute__((ext_vector_type(4)));

// buffer-load cache policy bits (gfx950): bit 1 = nontemporal
template <int POL>
__device__ __forceinline__ v4i probe_load(__amdgpu_buffer_rsrc_t r, int off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, POL);
}

template <int POL, int PASSES>
__global__ void __launch_bounds__(kProbeBlock) rs_probe_read_kernel(const char* __restrict__ src, int chunk_bytes,
                                                                    uint32_t* __restrict__ sink) {
    const char* base = src + (int64_t)blockIdx.x * chunk_bytes;
    // the descriptor covers exactly this workgroup's chunk
    const __amdgpu_buffer_rsrc_t r =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base), 0, chunk_bytes, 0x00020000);
    const int iters = chunk_bytes / kChunkQuantum;
    int acc = 0;
    for (int k = 0; k < iters; ++k) {
        v4i v[kProbeUnroll];
#pragma unroll
        for (int u = 0; u < kProbeUnroll; ++u)
            v[u] = probe_load<POL>(r, ((k * kProbeUnroll + u) * kProbeBlock + (int)threadIdx.x) * 16);
#pragma unroll
        for (int u = 0; u < kProbeUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    if (PASSES == 2) {
        __syncthreads();
        for (int k = iters - 1; k >= 0; --k) {
            v4i v[kProbeUnroll];
#pragma unroll
            for (int u = 0; u < kProbeUnroll; ++u)
                v[u] = probe_load<2>(r, ((k * kProbeUnroll + u) * kProbeBlock + (int)threadIdx.x) * 16);
#pragma unroll
            for (int u = 0; u < kProbeUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
        }
    }
    if (acc == 0x1234567) sink[blockIdx.x] = (uint32_t)acc;
}

template <int POL, int PASSES>
int launch_probe(const void* src, int64_t nchunks, int32_t chunk_bytes, void* sink, hipStream_t s) {
    hipLaunchKernelGGL((rs_probe_read_kernel<POL, PASSES>), dim3((unsigned)nchunks), dim3(kProbeBlock), 0, s,
                       static_cast<const char*>(src), chunk_bytes, static_cast<uint32_t*>(sink));
    return hipGetLastError() == hipSuccess ? 0 : 2;
}

}  // namespace

extern "C" int resispec_probe_read(const void* src, int64_t nbytes, int32_t chunk_bytes, int32_t policy,
                                   int32_t passes, void* sink, hipStream_t stream) {
    if (!src || !sink || nbytes <= 0 || chunk_bytes <= 0 || chunk_bytes % kChunkQuantum != 0 ||
        nbytes % chunk_bytes != 0 || (policy != 0 && policy != 1) || (passes != 1 && passes != 2))
        return 1;
    const int64_t nchunks = nbytes / chunk_bytes;
    if (nchunks >= (int64_t)1 << 31) return 1;
    if (policy == 0) return passes == 1 ? launch_probe<0, 1>(src, nchunks, chunk_bytes, sink, stream)
                                        : launch_probe<0, 2>(src, nchunks, chunk_bytes, sink, stream);
    return passes == 1 ? launch_probe<2, 1>(src, nchunks, chunk_bytes, sink, stream)
                       : launch_probe<2, 2>(src, nchunks, chunk_bytes, sink, stream);
}
