// Reference kernels for measurement, not part of the credit-assignment path: the streaming
// ceiling that a single-pass kernel with GAE's traffic can reach, and the cost of an empty
// launch. Built into libprobe.so, separately from librlcs.so.
//
// probe_stream_gae moves exactly the dense bytes of one GAE call with truncation per step:
// three 4-byte data inputs (rewards, values, truncation continuations) and two flag bytes read,
// two 4-byte outputs written, 22 bytes per step, with the same access shape as the GAE row
// kernel (one 16-byte non-temporal vector of each data array and one 4-byte word of each flag
// array per lane, 4 steps per lane). The arithmetic is a token one so that no load can be
// dropped; no scan, no dependence between lanes. probe_stream_gae_shape moves the same arrays in
// other launch shapes (workgroup size, vectors per lane, persistent grids) and optionally with
// the GAE kernel's dependent continuation loads, for the shape sweep of bench.py --probe-sweep.
#include <hip/hip_runtime.h>

#include <climits>
#include <cstdint>

typedef float f4 __attribute__((ext_vector_type(4)));

namespace {

// One lane streams `U` vectors, at i0, i0 + L, ..., i0 + (U-1) L (L = the grid's lanes), with
// every load of all U issued before the first store. kDep: the truncation continuation vector is
// loaded only when the lane's truncation word is nonzero, after the flag words arrive (the
// dependence the GAE kernel has); otherwise densely with the other data.
template <int kThreads, int U, bool kDep>
__global__ void __launch_bounds__(kThreads)
stream_gae_kernel(const f4* __restrict__ r, const f4* __restrict__ v, const f4* __restrict__ bv,
                  const uint32_t* __restrict__ term, const uint32_t* __restrict__ trunc,
                  f4* __restrict__ o0, f4* __restrict__ o1, int64_t n4) {
    const int64_t lanes = int64_t(gridDim.x) * kThreads;
    const int64_t i0 = int64_t(blockIdx.x) * kThreads + threadIdx.x;
    uint32_t te[U], tr[U];
    f4 a[U], b[U], c[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t i = i0 + u * lanes;
        if (i < n4) {
            te[u] = __builtin_nontemporal_load(term + i);
            tr[u] = __builtin_nontemporal_load(trunc + i);
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t i = i0 + u * lanes;
        if (i < n4) {
            a[u] = __builtin_nontemporal_load(r + i);
            b[u] = __builtin_nontemporal_load(v + i);
            if (!kDep) c[u] = __builtin_nontemporal_load(bv + i);
        }
    }
    if (kDep) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t i = i0 + u * lanes;
            c[u] = 0.f;
            if (i < n4 && tr[u]) c[u] = __builtin_nontemporal_load(bv + i);
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t i = i0 + u * lanes;
        if (i < n4) {
            const float s = ((te[u] | tr[u]) & 1u) ? 0.f : 1.f;
            __builtin_nontemporal_store(a[u] + b[u] * s, o0 + i);
            __builtin_nontemporal_store(c[u] + b[u], o1 + i);
        }
    }
}

// Persistent grid: each lane walks vectors i0, i0 + L, ... (L = the grid's lanes) with the next
// vector's loads issued before the current one's stores; every lane stops once past n4.
template <int kThreads>
__global__ void __launch_bounds__(kThreads)
stream_gae_persistent_kernel(const f4* __restrict__ r, const f4* __restrict__ v,
                             const f4* __restrict__ bv, const uint32_t* __restrict__ term,
                             const uint32_t* __restrict__ trunc, f4* __restrict__ o0,
                             f4* __restrict__ o1, int64_t n4) {
    const int64_t lanes = int64_t(gridDim.x) * kThreads;
    int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
    if (i >= n4) return;
    uint32_t te = __builtin_nontemporal_load(term + i), tr = __builtin_nontemporal_load(trunc + i);
    f4 a = __builtin_nontemporal_load(r + i), b = __builtin_nontemporal_load(v + i);
    f4 c = __builtin_nontemporal_load(bv + i);
    for (;;) {
        const int64_t j = i + lanes;
        const int64_t jc = j < n4 ? j : i;  // the last round reloads its own vector, unused
        const uint32_t nte = __builtin_nontemporal_load(term + jc), ntr = __builtin_nontemporal_load(trunc + jc);
        const f4 na = __builtin_nontemporal_load(r + jc), nb = __builtin_nontemporal_load(v + jc);
        const f4 nc = __builtin_nontemporal_load(bv + jc);
        __builtin_amdgcn_sched_barrier(0);
        const float s = ((te | tr) & 1u) ? 0.f : 1.f;
        __builtin_nontemporal_store(a + b * s, o0 + i);
        __builtin_nontemporal_store(c + b, o1 + i);
        if (j >= n4) break;
        i = j; te = nte; tr = ntr; a = na; b = nb; c = nc;
    }
}

__global__ void empty_kernel() {}

}  // namespace

extern "C" {

// Streams n steps (n a multiple of 4; every pointer 16-byte aligned, flags 4-byte aligned) in
// one of several launch shapes: workgroups of `threads` lanes (64 or 256); `per_lane` vectors of
// each array per lane (1, 2 or 4); `groups` = 0 for a grid that covers the array once, or the
// size of a persistent grid (with per_lane = 1) whose lanes walk the array; `dep` = 1 loads the
// truncation continuations only where the truncation word is nonzero (not with a persistent
// grid). Returns 0, 1 for bad arguments, 2 if the launch failed.
int probe_stream_gae_shape(const void* r, const void* v, const void* bv, const void* term,
                           const void* trunc, void* o0, void* o1, int64_t n, int threads,
                           int per_lane, int64_t groups, int dep, void* stream) {
    if (n < 0 || n % 4 != 0 || !r || !v || !bv || !term || !trunc || !o0 || !o1) return 1;
    for (const void* p : {r, v, bv, static_cast<const void*>(o0), static_cast<const void*>(o1)})
        if (reinterpret_cast<uintptr_t>(p) % 16) return 1;
    for (const void* p : {term, trunc})
        if (reinterpret_cast<uintptr_t>(p) % 4) return 1;
    if (threads != 64 && threads != 256) return 1;
    if (per_lane != 1 && per_lane != 2 && per_lane != 4) return 1;
    if (groups < 0 || groups > INT32_MAX || (groups > 0 && (per_lane != 1 || dep))) return 1;
    if (dep != 0 && dep != 1) return 1;
    const int64_t n4 = n / 4;
    if (n4 == 0) return 0;
    const int64_t per_group = int64_t(threads) * per_lane;
    const int64_t grid = groups > 0 ? groups : (n4 + per_group - 1) / per_group;
    if (grid > INT32_MAX) return 1;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const auto* rr = static_cast<const f4*>(r);
    const auto* vv = static_cast<const f4*>(v);
    const auto* bb = static_cast<const f4*>(bv);
    const auto* te = static_cast<const uint32_t*>(term);
    const auto* tr = static_cast<const uint32_t*>(trunc);
    auto* x = static_cast<f4*>(o0);
    auto* y = static_cast<f4*>(o1);
    const dim3 g(static_cast<unsigned>(grid)), b(static_cast<unsigned>(threads));
#define RLCS_PROBE(TH, U, DEP) \
    hipLaunchKernelGGL((stream_gae_kernel<TH, U, DEP>), g, b, 0, s, rr, vv, bb, te, tr, x, y, n4)
    if (groups > 0) {
        if (threads == 64)
            hipLaunchKernelGGL(stream_gae_persistent_kernel<64>, g, b, 0, s, rr, vv, bb, te, tr, x, y, n4);
        else
            hipLaunchKernelGGL(stream_gae_persistent_kernel<256>, g, b, 0, s, rr, vv, bb, te, tr, x, y, n4);
    } else if (threads == 64) {
        if (per_lane == 1) { if (dep) RLCS_PROBE(64, 1, true); else RLCS_PROBE(64, 1, false); }
        else if (per_lane == 2) { if (dep) RLCS_PROBE(64, 2, true); else RLCS_PROBE(64, 2, false); }
        else { if (dep) RLCS_PROBE(64, 4, true); else RLCS_PROBE(64, 4, false); }
    } else {
        if (per_lane == 1) { if (dep) RLCS_PROBE(256, 1, true); else RLCS_PROBE(256, 1, false); }
        else if (per_lane == 2) { if (dep) RLCS_PROBE(256, 2, true); else RLCS_PROBE(256, 2, false); }
        else { if (dep) RLCS_PROBE(256, 4, true); else RLCS_PROBE(256, 4, false); }
    }
#undef RLCS_PROBE
    return hipGetLastError() == hipSuccess ? 0 : 2;
}

// The dense streaming reference of bench.py's JSON line: one vector per lane, every array read.
int probe_stream_gae(const void* r, const void* v, const void* bv, const void* term,
                     const void* trunc, void* o0, void* o1, int64_t n, int threads, void* stream) {
    return probe_stream_gae_shape(r, v, bv, term, trunc, o0, o1, n, threads, 1, 0, 0, stream);
}

// One empty one-wave workgroup: the fixed cost of a launch in a stream or graph.
int probe_empty(void* stream) {
    hipLaunchKernelGGL(empty_kernel, dim3(1), dim3(64), 0, reinterpret_cast<hipStream_t>(stream));
    return hipGetLastError() == hipSuccess ? 0 : 2;
}

}  // extern "C"
