// Reference kernels for measurement, not part of the credit-assignment path: the streaming
// ceiling that a single-pass kernel with GAE's traffic can reach, and the cost of an empty
// launch. Built into libprobe.so, separately from librlcs.so.
//
// probe_stream_gae moves exactly the dense bytes of one GAE call with truncation per step:
// three 4-byte data inputs (rewards, values, truncation continuations) and two flag bytes read,
// two 4-byte outputs written, 22 bytes per step, with the same access shape as the GAE row
// kernel (one 16-byte non-temporal vector of each data array and one 4-byte word of each flag
// array per lane, 4 steps per lane). The arithmetic is a token one so that no load can be
// dropped; no scan, no dependence between lanes.
#include <hip/hip_runtime.h>

#include <cstdint>

typedef float f4 __attribute__((ext_vector_type(4)));

namespace {

template <int kThreads>
__global__ void __launch_bounds__(kThreads)
stream_gae_kernel(const f4* __restrict__ r, const f4* __restrict__ v, const f4* __restrict__ bv,
                  const uint32_t* __restrict__ term, const uint32_t* __restrict__ trunc,
                  f4* __restrict__ o0, f4* __restrict__ o1, int64_t n4) {
    const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
    if (i >= n4) return;
    const uint32_t te = __builtin_nontemporal_load(term + i);
    const uint32_t tr = __builtin_nontemporal_load(trunc + i);
    const f4 a = __builtin_nontemporal_load(r + i);
    const f4 b = __builtin_nontemporal_load(v + i);
    const f4 c = __builtin_nontemporal_load(bv + i);
    const float s = ((te | tr) & 1u) ? 0.f : 1.f;
    const f4 x = a + b * s;
    const f4 y = c + b;
    __builtin_nontemporal_store(x, o0 + i);
    __builtin_nontemporal_store(y, o1 + i);
}

__global__ void empty_kernel() {}

}  // namespace

extern "C" {

// Streams n steps (n a multiple of 4; every pointer 16-byte aligned, flags 4-byte aligned) with
// workgroups of `threads` lanes (64 or 256). Returns 0, or 1 for bad arguments, 2 if the launch
// failed.
int probe_stream_gae(const void* r, const void* v, const void* bv, const void* term,
                     const void* trunc, void* o0, void* o1, int64_t n, int threads, void* stream) {
    if (n < 0 || n % 4 != 0 || !r || !v || !bv || !term || !trunc || !o0 || !o1) return 1;
    for (const void* p : {r, v, bv, static_cast<const void*>(o0), static_cast<const void*>(o1)})
        if (reinterpret_cast<uintptr_t>(p) % 16) return 1;
    for (const void* p : {term, trunc})
        if (reinterpret_cast<uintptr_t>(p) % 4) return 1;
    if (threads != 64 && threads != 256) return 1;
    const int64_t n4 = n / 4;
    if (n4 == 0) return 0;
    const int64_t groups = (n4 + threads - 1) / threads;
    if (groups > INT32_MAX) return 1;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const auto* rr = static_cast<const f4*>(r);
    const auto* vv = static_cast<const f4*>(v);
    const auto* bb = static_cast<const f4*>(bv);
    const auto* te = static_cast<const uint32_t*>(term);
    const auto* tr = static_cast<const uint32_t*>(trunc);
    auto* x = static_cast<f4*>(o0);
    auto* y = static_cast<f4*>(o1);
    if (threads == 64)
        hipLaunchKernelGGL(stream_gae_kernel<64>, dim3(unsigned(groups)), dim3(64), 0, s, rr, vv, bb,
                           te, tr, x, y, n4);
    else
        hipLaunchKernelGGL(stream_gae_kernel<256>, dim3(unsigned(groups)), dim3(256), 0, s, rr, vv, bb,
                           te, tr, x, y, n4);
    return hipGetLastError() == hipSuccess ? 0 : 2;
}

// One empty one-wave workgroup: the fixed cost of a launch in a stream or graph.
int probe_empty(void* stream) {
    hipLaunchKernelGGL(empty_kernel, dim3(1), dim3(64), 0, reinterpret_cast<hipStream_t>(stream));
    return hipGetLastError() == hipSuccess ? 0 : 2;
}

}  // extern "C"
