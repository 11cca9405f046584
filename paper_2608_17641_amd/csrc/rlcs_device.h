// Device building blocks shared by every rlcs kernel: the affine pair and its composition
// (Eq. 2), the wave64 scan over lanes, and vectorised loads/stores of K consecutive elements.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rlcs {

constexpr int kWave = 64;

// An affine map X -> a + b * X. Composing the maps of consecutive steps is the combine of
// Eq. 2: the step nearer to the output position is `outer`, the one nearer to the carry
// source (later in time for backward scans, earlier for forward scans) is `inner`.
struct Pair {
    float a, b;
};

__device__ __forceinline__ Pair identity_pair() { return Pair{0.f, 1.f}; }

__device__ __forceinline__ Pair compose(Pair outer, Pair inner) {
    return Pair{fmaf(outer.b, inner.a, outer.a), outer.b * inner.b};
}

// Value of the map at X.
__device__ __forceinline__ float apply(Pair m, float x) { return fmaf(m.b, x, m.a); }

// DPP lane moves (GFX9 data-parallel primitives). A lane whose source lane does not exist
// keeps `fill`.
constexpr int kDppRowShr = 0x110;  // row_shr:n = 0x110 + n (within rows of 16 lanes)
constexpr int kDppWaveShr1 = 0x138;  // wave_shr:1 (lane i reads lane i-1 across the wave)

template <int kCtrl>
__device__ __forceinline__ float dpp_move(float fill, float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(fill), __float_as_int(v), kCtrl,
                                                      0xf, 0xf, false));
}

// Value of lane i-1 (lane 0 receives `fill`).
__device__ __forceinline__ float shift_up1(float v, float fill) { return dpp_move<kDppWaveShr1>(fill, v); }

__device__ __forceinline__ Pair read_lane(Pair v, int lane) {
    return Pair{__int_as_float(__builtin_amdgcn_readlane(__float_as_int(v.a), lane)),
                __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v.b), lane))};
}

// One Kogge-Stone step of the wave scan folded into two DPP-modified VALU operations: a lane
// whose DPP source lane exists (and is written by the row mask) composes its map with the
// source's map, the source inner: a += b * a_src, then b *= b_src. With bound_ctrl off, a lane
// whose source does not exist is not written and keeps its map, as composing with the identity
// would leave it. Each DPP read of a register a VALU operation wrote just before needs two wait
// states, hence the s_nop 1 ahead of each.
#define RLCS_DPP_STEP(v, CTRL)                                                             \
    asm volatile("s_nop 1\n\tv_fmac_f32_dpp %0, %0, %1 " CTRL " bank_mask:0xf\n\t"        \
                 "s_nop 1\n\tv_mul_f32_dpp %1, %1, %1 " CTRL " bank_mask:0xf"               \
                 : "+v"(v.a), "+v"(v.b))

// Inclusive prefix scan of per-lane maps over the 64 lanes (lane l ends with lanes 0..l
// composed, lane 0 innermost): Kogge-Stone inside each row of 16 lanes with DPP row shifts
// (4 steps, the tree of the Hillis-Steele trace of Appendix A), then two row broadcasts carry
// the row totals onto the rows after them. Twelve VALU operations, no LDS, no lane reads;
// moving the source maps into registers first (with the identity where a source is missing)
// and reading the row totals into scalars took 39.
__device__ __forceinline__ Pair wave_scan_inclusive(Pair v, int lane) {
    (void)lane;
    RLCS_DPP_STEP(v, "row_shr:1 row_mask:0xf");
    RLCS_DPP_STEP(v, "row_shr:2 row_mask:0xf");
    RLCS_DPP_STEP(v, "row_shr:4 row_mask:0xf");
    RLCS_DPP_STEP(v, "row_shr:8 row_mask:0xf");
    // rows 1 and 3 take lane 15 of the row before; then rows 2 and 3 take lane 31
    RLCS_DPP_STEP(v, "row_bcast:15 row_mask:0xa");
    RLCS_DPP_STEP(v, "row_bcast:31 row_mask:0xc");
    return v;
}
#undef RLCS_DPP_STEP

// ------------------------------------------------------------------ element loads / stores

// Element types of floating inputs: float, or bfloat16 held as its 16-bit pattern.
struct bf16_t {
    uint16_t bits;
};

__device__ __forceinline__ float widen(float x) { return x; }
__device__ __forceinline__ float widen(bf16_t x) { return __uint_as_float(uint32_t(x.bits) << 16); }

template <typename DT>
__device__ __forceinline__ float load_one(const void* base, int64_t i) {
    return widen(reinterpret_cast<const DT*>(base)[i]);
}

// Raw 32-bit words -> K widened values.
template <typename DT, int K>
__device__ __forceinline__ void unpack_words(const uint32_t* w, float (&out)[K]) {
    if constexpr (sizeof(DT) == 4) {
#pragma unroll
        for (int k = 0; k < K; ++k) out[k] = __uint_as_float(w[k]);
    } else {
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const uint32_t word = w[k >> 1];
            out[k] = __uint_as_float((k & 1) ? (word & 0xffff0000u) : (word << 16));
        }
    }
}

// Element k of the DT values packed in a 32-bit word holding element `k` of a block (fp32: the
// word itself; bf16: the low half for even k, the high half for odd k).
template <typename DT>
__device__ __forceinline__ float word_elem(uint32_t word, int k) {
    if constexpr (sizeof(DT) == 4) return __uint_as_float(word);
    else return __uint_as_float((k & 1) ? (word & 0xffff0000u) : (word << 16));
}

// K consecutive elements starting at p0 (a multiple of K). `full`: all K are in range and the
// pointer is 16-byte aligned, so the load is one or more 16-byte vector loads. Otherwise only
// elements whose bit is set in `valid` are read; the rest are 0.
template <typename DT, int K>
__device__ __forceinline__ void load_k(const void* base, int64_t p0, uint32_t valid, bool full,
                                       float (&out)[K]) {
    constexpr int kBytes = K * int(sizeof(DT));
    static_assert(kBytes % 16 == 0 || kBytes == 8, "vector width");
    if (full) {
        uint32_t w[kBytes / 4];
        const char* p = reinterpret_cast<const char*>(base) + p0 * int64_t(sizeof(DT));
        if constexpr (kBytes % 16 == 0) {
#pragma unroll
            for (int i = 0; i < kBytes / 16; ++i) {
                const uint4 u = reinterpret_cast<const uint4*>(p)[i];
                w[4 * i + 0] = u.x; w[4 * i + 1] = u.y; w[4 * i + 2] = u.z; w[4 * i + 3] = u.w;
            }
        } else {
            const uint2 u = *reinterpret_cast<const uint2*>(p);
            w[0] = u.x; w[1] = u.y;
        }
        unpack_words<DT, K>(w, out);
    } else {
#pragma unroll
        for (int k = 0; k < K; ++k)
            out[k] = ((valid >> k) & 1u) ? load_one<DT>(base, p0 + k) : 0.f;
    }
}

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));

// Flags of K consecutive steps: raw 32-bit words (vector path) and their K-bit mask (bit k
// set: byte k nonzero). Loading and converting are separate so that every load of a chunk can
// be issued before the first use of any of them. Non-temporal: each flag is read once.
template <int K>
__device__ __forceinline__ void load_flag_words(const uint8_t* base, int64_t p0, uint32_t (&w)[(K + 3) / 4]) {
    if constexpr (K == 4) {
        w[0] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(base + p0));
    } else if constexpr (K == 8) {
        const u32x2 u = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(base + p0));
        w[0] = u.x; w[1] = u.y;
    } else {
        static_assert(K == 16, "flag vector width");
        const u32x4 u = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(base + p0));
        w[0] = u.x; w[1] = u.y; w[2] = u.z; w[3] = u.w;
    }
}

template <int K>
__device__ __forceinline__ uint32_t flag_mask(const uint32_t (&w)[(K + 3) / 4]) {
    uint32_t m = 0;
#pragma unroll
    for (int k = 0; k < K; ++k) m |= (((w[k >> 2] >> (8 * (k & 3))) & 0xffu) != 0u) ? (1u << k) : 0u;
    return m;
}

// Masked element-wise flag load (ragged chunks).
template <int K>
__device__ __forceinline__ uint32_t load_flags_masked(const uint8_t* base, int64_t p0, uint32_t valid) {
    uint32_t m = 0;
#pragma unroll
    for (int k = 0; k < K; ++k)
        if ((valid >> k) & 1u) m |= (base[p0 + k] != 0) ? (1u << k) : 0u;
    return m;
}

// Raw words of K consecutive data elements: 16-byte vector loads, non-temporal because every
// input is read exactly once.
template <typename DT, int K>
__device__ __forceinline__ void load_words(const void* base, int64_t p0, uint32_t (&w)[K * sizeof(DT) / 4]) {
    constexpr int kBytes = K * int(sizeof(DT));
    static_assert(kBytes % 16 == 0 || kBytes == 8, "vector width");
    const char* p = reinterpret_cast<const char*>(base) + p0 * int64_t(sizeof(DT));
    if constexpr (kBytes % 16 == 0) {
#pragma unroll
        for (int i = 0; i < kBytes / 16; ++i) {
            const u32x4 u = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p) + i);
            w[4 * i + 0] = u.x; w[4 * i + 1] = u.y; w[4 * i + 2] = u.z; w[4 * i + 3] = u.w;
        }
    } else {
        const u32x2 u = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p));
        w[0] = u.x; w[1] = u.y;
    }
}

typedef float f32x4 __attribute__((ext_vector_type(4)));

// Outputs are written once and not read again by the kernel: non-temporal 16-byte stores.
template <int K>
__device__ __forceinline__ void store_k(float* base, int64_t p0, uint32_t valid, bool full,
                                        const float (&v)[K]) {
    if (full) {
        f32x4* p = reinterpret_cast<f32x4*>(base + p0);
#pragma unroll
        for (int i = 0; i < K / 4; ++i) {
            const f32x4 q = {v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]};
            __builtin_nontemporal_store(q, p + i);
        }
    } else {
#pragma unroll
        for (int k = 0; k < K; ++k)
            if ((valid >> k) & 1u) base[p0 + k] = v[k];
    }
}

// Lanes of one wave exchanging values through LDS: every LDS write of the wave before the call
// is seen by every LDS read after it (a wave's LDS instructions run in issue order; the fences
// keep the compiler from moving LDS accesses across the call).
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Eight outputs per lane (K = 8: bf16 inputs) where the wave's outputs are the 512 consecutive
// ones [base, base + 512) and lane l holds group g of them. As two 16-byte stores per lane,
// each store instruction of the wave would cover every other 16 bytes of its 2 KB, and
// non-temporal stores of such half lines reach HBM as whole lines (6-11 % of the lines written
// twice). Through the wave's 2 KB LDS `slot` lane l stores 16-byte pieces l and 64 + l instead,
// so that each store instruction covers 1 KB of whole 128-byte lines. Pieces at or past `limit`
// (a multiple of 8) are not stored. Every lane of the wave takes part; `out + base` is 16-byte
// aligned.
__device__ __forceinline__ void store8_lines(float* out, int64_t base, int64_t limit, int g,
                                             int lane, const float (&v)[8], f32x4* slot) {
    wave_lds_sync();  // the slot's previous readers are done
    slot[2 * g] = f32x4{v[0], v[1], v[2], v[3]};
    slot[2 * g + 1] = f32x4{v[4], v[5], v[6], v[7]};
    wave_lds_sync();
    const f32x4 x0 = slot[lane], x1 = slot[kWave + lane];
    const int64_t p = base + 4 * int64_t(lane);
    if (p < limit) __builtin_nontemporal_store(x0, reinterpret_cast<f32x4*>(out + p));
    if (p + 4 * kWave < limit)
        __builtin_nontemporal_store(x1, reinterpret_cast<f32x4*>(out + p + 4 * kWave));
}

}  // namespace rlcs
