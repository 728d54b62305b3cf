// Cross-XCD coherence litmus test of the in-launch exchange the persistent,
// dataflow and resident drivers rely on: a producer workgroup stores a block
// with agent-coherent (sc1) buffer stores, waits for them to land
// (s_waitcnt), and bumps a counter with a relaxed agent-scope atomic; a
// consumer workgroup on another XCD polls the counter (bounded), then reads
// the block and checks every value.  Mode 0 reads with agent-coherent loads
// (the persistent and dataflow drivers, which reuse buffers); mode 1 with
// ordinary cached loads of addresses written once per launch (the resident
// driver's per-task buffers); mode 2 bumps the counter as soon as the stores
// are issued (no s_waitcnt) and the consumer, on a block filled with an
// all-ones word before the launch, reads agent-coherent and reads again every
// word that still holds the fill (the resident driver's fp32 h1 and h2).
#include "wf_device.h"

namespace wf {

constexpr int kLitmusWords = 1024;   // words of one block (4 per thread)

constexpr unsigned kLitmusFill = 0xFFFFFFFFu;   // mode 2's fill word (no value below is one)

__device__ __forceinline__ unsigned litmus_value(int round, int pair, int i) {
    return ((unsigned)round * 2654435761u ^ (unsigned)pair * 40503u ^ (unsigned)i * 97u ^ 0x5bd1e995u) & 0x7FFFFFFFu;
}

// Workgroups [0, npair) produce, [npair, 2 npair) consume; consumer q reads
// what producer (q + 1) mod npair wrote, which sits on another XCD when
// workgroups are dealt to the XCDs round robin.  data: [npair][rounds][1024]
// words, cnt: [npair][rounds] counters (zero before the launch).
__global__ __launch_bounds__(kThreads) void k_litmus(unsigned* data, unsigned* cnt, int npair, int rounds, int mode,
                                                     unsigned* bad, int* err, long long budget) {
    __shared__ int bail;
    const int g = blockIdx.x;
    const bool prod = g < npair;
    const int pair = prod ? g : (g - npair + 1) % npair;
    for (int r = 0; r < rounds; ++r) {
        unsigned* blk = data + ((size_t)pair * rounds + r) * kLitmusWords;
        unsigned* c = cnt + (size_t)pair * rounds + r;
        if (prod) {
            for (int i = threadIdx.x; i < kLitmusWords; i += blockDim.x)
                st1<true>(reinterpret_cast<float*>(blk), i, __builtin_bit_cast(float, litmus_value(r, pair, i)));
            if (mode != 2) __builtin_amdgcn_s_waitcnt(0);
            __builtin_amdgcn_s_barrier();
            if (threadIdx.x == 0) __hip_atomic_fetch_add(c, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            continue;
        }
        if (threadIdx.x == 0) {
            int flag = 0;
            const long long t0 = wall_clock64();
            while (__hip_atomic_load(c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < 1u) {
                if (__hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0 ||
                    wall_clock64() - t0 > budget) {
                    __hip_atomic_store(err, kErrTimeout, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    flag = 1;
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
            bail = flag;
        }
        __syncthreads();
        if (bail) return;
        unsigned nbad = 0;
        for (int i = threadIdx.x; i < kLitmusWords; i += blockDim.x) {
            const float* b = reinterpret_cast<const float*>(blk);
            float v = mode == 1 ? ld1<false>(b, i) : ld1<true>(b, i);
            if (mode == 2) {
                const long long t0 = wall_clock64();
                while (__builtin_bit_cast(unsigned, v) == kLitmusFill && wall_clock64() - t0 <= budget) {
                    __builtin_amdgcn_s_sleep(1);
                    v = ld1<true>(b, i);
                }
            }
            nbad += __builtin_bit_cast(unsigned, v) != litmus_value(r, pair, i);
        }
        if (nbad) atomicAdd(bad, nbad);
    }
}

__global__ void k_litmus_zero(unsigned* p, size_t n, unsigned v = 0u) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = v;
}

}  // namespace wf

using namespace wf;

extern "C" int wf_litmus(int32_t mode, int32_t pairs, int32_t rounds, uint64_t* mismatches, hipStream_t stream) {
    if (!mismatches || mode < 0 || mode > 2 || pairs < 1 || rounds < 1)
        return fail(WF_E_INVALID, "mode must be 0, 1 or 2, pairs and rounds positive, mismatches non-NULL");
    const size_t words = (size_t)pairs * rounds * kLitmusWords;
    if (words * 4 >= (size_t)kBufBytes) return fail(WF_E_INVALID, "pairs x rounds too large for one buffer");
    int dev = 0, cus = 0, per_cu = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, (const void*)k_litmus, kThreads, 0);
    if (e != hipSuccess) return fail(WF_E_HIP, std::string("device query: ") + hipGetErrorString(e));
    if (2 * pairs > cus * per_cu) return fail(WF_E_UNSUPPORTED, "too many pairs to be resident at once");
    unsigned *data = nullptr, *cnt = nullptr, *bad = nullptr;
    int* err = nullptr;
    auto cleanup = [&]() {
        if (data) (void)hipFree(data);
        if (cnt) (void)hipFree(cnt);
        if (bad) (void)hipFree(bad);
        if (err) (void)hipFree(err);
    };
    e = hipMalloc((void**)&data, words * 4);
    if (e == hipSuccess) e = hipMalloc((void**)&cnt, (size_t)pairs * rounds * 4 + 4);
    if (e == hipSuccess) e = hipMalloc((void**)&bad, 4);
    if (e == hipSuccess) e = hipMalloc((void**)&err, 4);
    if (e != hipSuccess) {
        cleanup();
        return fail(WF_E_NOMEM, std::string("litmus buffers: ") + hipGetErrorString(e));
    }
    hipLaunchKernelGGL(k_litmus_zero, dim3(256), dim3(256), 0, stream, data, words, mode == 2 ? kLitmusFill : 0u);
    hipLaunchKernelGGL(k_litmus_zero, dim3(64), dim3(256), 0, stream, cnt, (size_t)pairs * rounds, 0u);
    hipLaunchKernelGGL(k_litmus_zero, dim3(1), dim3(64), 0, stream, bad, (size_t)1, 0u);
    hipLaunchKernelGGL(k_litmus_zero, dim3(1), dim3(64), 0, stream, reinterpret_cast<unsigned*>(err), (size_t)1, 0u);
    int np = pairs, nr = rounds, md = mode;
    long long budget = 100000000;   // 1 s of wall clock (100 MHz)
    void* args[] = {&data, &cnt, &np, &nr, &md, &bad, &err, &budget};
    e = hipLaunchCooperativeKernel((const void*)k_litmus, dim3(2 * pairs), dim3(kThreads), args, 0, stream);
    unsigned hb = 0;
    int he = 0;
    if (e == hipSuccess) e = hipMemcpyAsync(&hb, bad, 4, hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipMemcpyAsync(&he, err, 4, hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    cleanup();
    if (e != hipSuccess) return fail(WF_E_HIP, std::string("litmus: ") + hipGetErrorString(e));
    *mismatches = hb;
    if (he) return fail(WF_E_TIMEOUT, "litmus: a consumer waited longer than its budget");
    return WF_OK;
}
