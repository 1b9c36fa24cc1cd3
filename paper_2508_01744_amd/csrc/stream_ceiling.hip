// The attainable HBM rate of a step's memory traffic without its arithmetic,
// as the bound to read a step kernel's achieved rate against.
//
// One workgroup of 256 threads per instance, each over its own region of C
// 16-byte chunks (the instance's arm records), as the step kernel is laid
// out.  Two forms, timed in turn:
//   read:            every chunk of the region read once with non-temporal
//                    loads (the records a step streams);
//   read+writeback:  the same, then R chunks (one record) written back with
//                    non-temporal stores at a record position inside the
//                    region that varies over instances (the update of the
//                    decided arm), as the last act of the workgroup.
// The pair separates the rate of the stream itself from the cost that the
// per-instance write-back adds to it.
//
// Built as its own library (libagft_ceiling.so), apart from the tuner's:
//   int agft_stream_ceiling_at(int64_t instances, int64_t chunks, int32_t record_chunks,
//                              int32_t launches, int32_t cu_workgroups,
//                              double *read_us, double *read_writeback_us)
// allocates a zero-filled buffer of instances x chunks x 16 bytes on the
// current device, times each form over `launches` launches on the null
// stream (after two untimed ones), writes the average duration of each in
// microseconds and frees the buffer.  cu_workgroups > 0 caps the workgroups
// per compute unit by the launches' LDS request (a 1/cap share of the unit's
// LDS, confirmed by the occupancy calculator), since the rate of concurrent
// streams depends on how many run at once; 0 leaves them uncapped.
// agft_stream_ceiling(...) without cu_workgroups is the uncapped form.
// Returns 0; 1 for arguments out of range (instances and chunks in [1, 2^31),
// record_chunks in [1, 256] and <= chunks, launches >= 1, cu_workgroups in
// [0, 64]); 2 for a HIP error (reported on stderr); 3 for a cap the
// occupancy calculator does not confirm.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>

namespace {

constexpr int kThreads = 256;
constexpr int kInFlight = 8;   // loads per thread issued before any is used

typedef float f4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f4 load_nt(const f4 *p) { return __builtin_nontemporal_load(p); }

template <bool WRITEBACK>
__global__ __launch_bounds__(kThreads) void stream_kernel(f4 *base, int chunks, int rec, float *sink) {
    f4 *region = base + (size_t)blockIdx.x * (size_t)chunks;
    const int tid = threadIdx.x;
    constexpr int kRound = kInFlight * kThreads;
    float acc = 0.0f;
    // whole rounds without bounds checks, so that every load of a round is
    // issued before any is used; then the rest, one chunk per thread at a time
    const int full = chunks / kRound * kRound;
    for (int c0 = 0; c0 < full; c0 += kRound) {
        f4 v[kInFlight];
#pragma unroll
        for (int u = 0; u < kInFlight; ++u) v[u] = load_nt(region + c0 + u * kThreads + tid);
#pragma unroll
        for (int u = 0; u < kInFlight; ++u) acc += (v[u].x + v[u].y) + (v[u].z + v[u].w);
    }
    for (int c = full + tid; c < chunks; c += kThreads) {
        const f4 v = load_nt(region + c);
        acc += (v.x + v.y) + (v.z + v.w);
    }
    if constexpr (WRITEBACK) {
        // a record position that varies over instances, inside the region
        const int nrec = chunks / rec;
        const int pos = (int)((blockIdx.x * 37u + 11u) % (unsigned)nrec) * rec;
        __syncthreads();
        if (tid < rec) __builtin_nontemporal_store((f4){acc, 1.0f, 2.0f, 3.0f}, region + pos + tid);
    }
    // keeps the loads live; the sum of a zero-filled region never matches
    if (acc == 1234.5f) sink[blockIdx.x] = acc;
}

bool ok(hipError_t e, const char *what) {
    if (e == hipSuccess) return true;
    std::fprintf(stderr, "agft_stream_ceiling: %s: %s\n", what, hipGetErrorString(e));
    return false;
}

// Dynamic LDS per workgroup that admits exactly `cap` workgroups of the
// kernel per compute unit (0 when cap is 0); -1 if none does.
int64_t cap_lds(const void *kernel, int cap) {
    if (cap == 0) return 0;
    int dev = 0, per_cu = 0;
    hipFuncAttributes fa;
    if (!ok(hipGetDevice(&dev), "hipGetDevice") ||
        !ok(hipDeviceGetAttribute(&per_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev), "attribute") ||
        !ok(hipFuncGetAttributes(&fa, kernel), "hipFuncGetAttributes"))
        return -2;
    const int64_t max_dyn = 64 * 1024 - (int64_t)fa.sharedSizeBytes;
    for (int64_t d = ((int64_t)per_cu / cap - (int64_t)fa.sharedSizeBytes) / 16 * 16; d > 0; d -= 512) {
        if (d > max_dyn) continue;
        int blocks = 0;
        if (!ok(hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, kernel, kThreads, (size_t)d), "occupancy"))
            return -2;
        if (blocks == cap) return d;
        if (blocks > cap) break;
    }
    return -1;
}

}  // namespace

extern "C" int agft_stream_ceiling_at(int64_t inst, int64_t chunks, int32_t rec, int32_t launches,
                                      int32_t cu_workgroups, double *read_us, double *read_writeback_us) {
    if (inst < 1 || inst > 0x7fffffffL || chunks < 1 || chunks > 0x7fffffffL || rec < 1 || rec > kThreads ||
        rec > chunks || launches < 1 || cu_workgroups < 0 || cu_workgroups > 64 || read_us == nullptr ||
        read_writeback_us == nullptr)
        return 1;
    int64_t lds[2];
    lds[0] = cap_lds(reinterpret_cast<const void *>(&stream_kernel<false>), cu_workgroups);
    lds[1] = cap_lds(reinterpret_cast<const void *>(&stream_kernel<true>), cu_workgroups);
    if (lds[0] == -2 || lds[1] == -2) return 2;
    if (lds[0] < 0 || lds[1] < 0) return 3;
    const size_t bytes = (size_t)inst * (size_t)chunks * 16;
    f4 *buf = nullptr;
    float *sink = nullptr;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    int rc = 0;
    if (!ok(hipMalloc(&buf, bytes), "hipMalloc") || !ok(hipMalloc(&sink, (size_t)inst * 4), "hipMalloc") ||
        !ok(hipMemset(buf, 0, bytes), "hipMemset") || !ok(hipEventCreate(&e0), "hipEventCreate") ||
        !ok(hipEventCreate(&e1), "hipEventCreate"))
        rc = 2;
    double *out[2] = {read_us, read_writeback_us};
    for (int form = 0; form < 2 && rc == 0; ++form) {
        auto launch = [&]() {
            if (form == 0)
                hipLaunchKernelGGL(stream_kernel<false>, dim3((unsigned)inst), dim3(kThreads), (size_t)lds[0], 0, buf,
                                   (int)chunks, (int)rec, sink);
            else
                hipLaunchKernelGGL(stream_kernel<true>, dim3((unsigned)inst), dim3(kThreads), (size_t)lds[1], 0, buf,
                                   (int)chunks, (int)rec, sink);
        };
        launch();
        launch();
        float ms = 0.0f;
        if (!ok(hipGetLastError(), "launch") || !ok(hipDeviceSynchronize(), "warm-up") || !ok(hipEventRecord(e0, 0), "hipEventRecord")) {
            rc = 2;
            break;
        }
        for (int q = 0; q < launches; ++q) launch();
        if (!ok(hipEventRecord(e1, 0), "hipEventRecord") || !ok(hipEventSynchronize(e1), "launches") ||
            !ok(hipEventElapsedTime(&ms, e0, e1), "hipEventElapsedTime")) {
            rc = 2;
            break;
        }
        *out[form] = (double)ms * 1e3 / launches;
    }
    if (e0 != nullptr) (void)hipEventDestroy(e0);
    if (e1 != nullptr) (void)hipEventDestroy(e1);
    if (buf != nullptr) (void)hipFree(buf);
    if (sink != nullptr) (void)hipFree(sink);
    return rc;
}

extern "C" int agft_stream_ceiling(int64_t inst, int64_t chunks, int32_t rec, int32_t launches, double *read_us,
                                   double *read_writeback_us) {
    return agft_stream_ceiling_at(inst, chunks, rec, launches, 0, read_us, read_writeback_us);
}
