// Eligibility traces of F-vectors along rows (Section 3.3.5): z_t = beta_t z_{t-1} + x_t for
// x_t, z_t in R^F, beta_t = gamma lambda except 0 at a row's first step and after a step that
// ends an episode, one beta per step shared by all F features.
//
// For F a multiple of the 16-byte vector width V (4 float32 or 8 bfloat16 features) with
// L = F / V lanes per step a power of two up to 64, one workgroup of W waves scans R whole rows
// of the [N, T, F] input as one range of R * T steps (contiguous in memory; the beta = 0 of each
// row's first step keeps rows apart, so the scan needs no other boundary). Lane l of wave w
// holds features [V (l mod L), V (l mod L) + V) of the kVecSteps = 4 consecutive steps from
// t0 = (w S + l / L) * 4 of the range, S = 64 / L step groups side by side in a wave. The wave's
// inputs and outputs, S * 4 consecutive steps, are contiguous: where a step is under 128 bytes
// (L < 8), each wave loads its inputs as whole 1 KB runs into its LDS slot, from which each lane
// takes one 16-byte vector per step (read straight from memory, half a line per step at F = 16
// float32: 4096 x 256 x 16 30.8 us against 27.0 staged; at F = 64 direct loads of whole lines
// 26.2 us against 27.2 staged). A lane's map over its steps is V offsets and one shared factor;
// a wave scans its step groups by shuffles across lanes L apart (log2 S rounds), the waves
// compose once through LDS (wave w's total maps at [w][F] offsets and [w] factors) and each lane
// finishes its steps. The outputs pass back through the slot so that each store instruction
// writes 1 KB of whole lines (pieces past the range's end are neither loaded nor stored). Flags:
// one 4-byte word per lane and array when `word_flags` (T a multiple of 4, aligned flag arrays),
// otherwise one byte per step; lanes also read the flags of the step before t0. Grid:
// ceil(N / R) workgroups of W * 64 lanes.
#pragma once

#include "rlcs_dispatch.h"

namespace rlcs {

constexpr int kVecSteps = 4;

// Bytes of dynamic LDS for a workgroup of W waves: W output slots of 64 * 4 * V floats, then
// W * F offsets and W factors.
template <typename DT>
constexpr size_t vec_rows_lds(int W, int64_t F) {
    constexpr int V = 16 / int(sizeof(DT));
    return size_t(W) * kWave * kVecSteps * V * 4 + size_t(W) * size_t(F) * 4 + size_t(W) * 4;
}

// Eight waves per SIMD for float32 inputs with L > 1 (the compiler keeps the kernel within 64
// VGPRs, no spills; left to itself it took 74-82 and ran 5 waves): fp32 4096 x 256 x 16
// 26.5 -> 25.7 us, 65536 x 8 x 16 15.4 -> 13.0, 2048 x 1024 x 16 64.8 -> 58.7, 1024 x 2048 x 8
// 35.5 -> 31.9. bfloat16 inputs and L = 1 stay unconstrained: held to 64 VGPRs they spill.
template <typename DT, int L>
constexpr int vec_rows_waves_per_eu() { return sizeof(DT) == 4 && L > 1 ? 8 : 1; }

template <typename DT, bool TR, int L>
__global__ void __launch_bounds__(16 * kWave) __attribute__((amdgpu_waves_per_eu(vec_rows_waves_per_eu<DT, L>())))
vec_rows_kernel(Args a, int R, int word_flags) {
    constexpr int V = 16 / int(sizeof(DT));
    constexpr int F = L * V;
    constexpr int S = kWave / L;
    constexpr int KS = kVecSteps;
    constexpr int kPieces = kWave * KS * V / 4;  // 16-byte output pieces of one wave
    extern __shared__ f32x4 s_vec[];
    const int W = int(blockDim.x) / kWave;
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    const int fg = lane % L, sg = lane / L;
    // the workgroup's rows [row0, row0 + R) as one range of E steps (a row's first step has
    // beta = 0, so the scan needs no other row boundary)
    const int64_t T = a.T;
    const int64_t row0 = int64_t(blockIdx.x) * R;
    const int64_t E = (min(row0 + R, a.N) - row0) * T;
    const int64_t frow = row0 * T;  // the range's first flag
    const int64_t xrow = frow * F;  // the range's first feature value
    const int t0 = (wave * S + sg) * KS;  // the lane's first step in the range
    float* s_off = reinterpret_cast<float*>(s_vec + W * kPieces);
    float* s_fac = s_off + W * F;
    const float decay = a.p.gamma * a.p.lambda;

    // loads, all issued before the first use: the lane's inputs, then its flags and those of the
    // step before t0. Steps of fewer than 128 bytes (L < 8) are staged: the wave loads its span,
    // S * KS consecutive steps of the range, as whole 1 KB runs (16-byte piece i * 64 + lane, up
    // to the range's end) into its slot, and each lane takes its pieces from there; longer steps
    // are whole lines already and each lane loads its own vectors.
    constexpr bool kStaged = L < 8;
    f32x4* slot = s_vec + wave * kPieces;
    const int64_t wbase = xrow + int64_t(wave) * S * KS * F;  // the wave's first element
    const int64_t limit = xrow + E * F;                       // the range's end
    const DT* x = static_cast<const DT*>(a.in[0]);
    int nv = 0;  // the lane's steps inside the range
    if (t0 < E) nv = int(min(int64_t(KS), E - t0));
    u32x4 raw[KS];
#pragma unroll
    for (int i = 0; i < KS; ++i) {
        const int64_t p = kStaged ? wbase + int64_t(i * kWave + lane) * V : xrow + (t0 + i) * F + fg * V;
        if (kStaged ? p < limit : i < nv)
            raw[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(x + p));
    }
    uint32_t done = 0;  // bit k: step t0 + k ends an episode
    bool cut0 = true;   // nothing enters step t0 (a row start, or an episode ended before it)
    const int r0 = t0 % int(T);  // step t0's place in its row
    if (t0 < E) {
        if (word_flags) {
            uint32_t tw[1] = {0u}, rw[1] = {0u};
            if (a.term) load_flag_words<4>(a.term, frow + t0, tw);
            if (TR) load_flag_words<4>(a.trunc, frow + t0, rw);
            done = flag_mask<4>(tw) | flag_mask<4>(rw);
        } else {
#pragma unroll
            for (int k = 0; k < KS; ++k) {
                if (k < nv) {
                    const bool d = (a.term && a.term[frow + t0 + k]) || (TR && a.trunc[frow + t0 + k]);
                    done |= d ? (1u << k) : 0u;
                }
            }
        }
        if (r0 > 0) cut0 = (a.term && a.term[frow + t0 - 1]) || (TR && a.trunc[frow + t0 - 1]);
    }
    if constexpr (kStaged) {
#pragma unroll
        for (int i = 0; i < KS; ++i) {
            const int64_t p = wbase + int64_t(i * kWave + lane) * V;
            if (p < limit) reinterpret_cast<u32x4*>(slot)[i * kWave + lane] = raw[i];
        }
        // the lane's vectors: step k's features at piece (sg * KS + k) * L + fg of the span
        wave_lds_sync();
#pragma unroll
        for (int k = 0; k < KS; ++k) raw[k] = reinterpret_cast<const u32x4*>(slot)[(sg * KS + k) * L + fg];
    }
    float xv[KS][V];
#pragma unroll
    for (int k = 0; k < KS; ++k) {
        const uint32_t w[4] = {raw[k].x, raw[k].y, raw[k].z, raw[k].w};
        if (k < nv) {
            unpack_words<DT, V>(w, xv[k]);
        } else {
#pragma unroll
            for (int v = 0; v < V; ++v) xv[k][v] = 0.f;
        }
    }

    // the lane's map over its steps: A_out = off + fac * A_in (steps past the row end are the
    // identity; they follow every step of the row)
    float be[KS];
    int r = r0;  // step t0 + k's place in its row
#pragma unroll
    for (int k = 0; k < KS; ++k) {
        const bool cut = k == 0 ? cut0 : (r == 0 || bit(done, k - 1));
        be[k] = k < nv ? (cut ? 0.f : decay) : 1.f;
        r = r + 1 == int(T) ? 0 : r + 1;
    }
    float off[V];
    float fac = be[0];
#pragma unroll
    for (int v = 0; v < V; ++v) off[v] = xv[0][v];
#pragma unroll
    for (int k = 1; k < KS; ++k) {
#pragma unroll
        for (int v = 0; v < V; ++v) off[v] = fmaf(be[k], off[v], xv[k][v]);
        fac *= be[k];
    }

    // the wave's step groups: inclusive scan over lanes L apart, then the map of the groups
    // before this lane's
    float eo[V], ef = 1.f;
#pragma unroll
    for (int v = 0; v < V; ++v) eo[v] = 0.f;
    if constexpr (S > 1) {
#pragma unroll
        for (int d = 1; d < S; d <<= 1) {
            float po[V];
#pragma unroll
            for (int v = 0; v < V; ++v) po[v] = __shfl_up(off[v], d * L);
            const float pf = __shfl_up(fac, d * L);
            if (sg >= d) {
#pragma unroll
                for (int v = 0; v < V; ++v) off[v] = fmaf(fac, po[v], off[v]);
                fac *= pf;
            }
        }
        float po[V];
#pragma unroll
        for (int v = 0; v < V; ++v) po[v] = __shfl_up(off[v], L);
        const float pf = __shfl_up(fac, L);
        if (sg > 0) {
#pragma unroll
            for (int v = 0; v < V; ++v) eo[v] = po[v];
            ef = pf;
        }
    }

    // the waves before this one, composed from the row start
    if (sg == S - 1) {
#pragma unroll
        for (int v = 0; v < V; ++v) s_off[wave * F + fg * V + v] = off[v];
        if (fg == 0) s_fac[wave] = fac;
    }
    __syncthreads();
    float X[V];
#pragma unroll
    for (int v = 0; v < V; ++v) X[v] = 0.f;
    for (int j = 0; j < wave; ++j) {
        const float f = s_fac[j];
#pragma unroll
        for (int v = 0; v < V; ++v) X[v] = fmaf(f, X[v], s_off[j * F + fg * V + v]);
    }
#pragma unroll
    for (int v = 0; v < V; ++v) X[v] = fmaf(ef, X[v], eo[v]);

    // the lane's steps, into the wave's slot (every lane of the wave has read its inputs from
    // it): step k's features at float offset (sg * KS + k) * F + fg * V of the wave's outputs
    wave_lds_sync();
#pragma unroll
    for (int k = 0; k < KS; ++k) {
#pragma unroll
        for (int v = 0; v < V; ++v) X[v] = fmaf(be[k], X[v], xv[k][v]);
        const int piece = ((sg * KS + k) * F + fg * V) / 4;
#pragma unroll
        for (int i = 0; i < V / 4; ++i)
            slot[piece + i] = f32x4{X[4 * i], X[4 * i + 1], X[4 * i + 2], X[4 * i + 3]};
    }
    wave_lds_sync();
#pragma unroll
    for (int i = 0; i < kPieces / kWave; ++i) {
        const int pc = i * kWave + lane;
        const int64_t p = wbase + 4 * int64_t(pc);
        if (p < limit) __builtin_nontemporal_store(slot[pc], reinterpret_cast<f32x4*>(a.out0 + p));
    }
}

namespace host {

// Fewest workgroups of the row kernel: with fewer, the column scans, which also split time, fill
// the GPU better.
constexpr int64_t kVecRowsMinGroups = 256;
// Dynamic LDS of one workgroup at most (the waves of a row are capped by it): what one CU of
// the MI355X holds, 160 KB.
constexpr size_t kVecRowsMaxLds = 160 * 1024;

template <typename DT, bool TR, int L>
void vec_rows_launch_l(const Args& a, int64_t groups, int W, int R, int word_flags, hipStream_t s) {
    hipLaunchKernelGGL((vec_rows_kernel<DT, TR, L>), dim3(unsigned(groups)), dim3(unsigned(W * kWave)),
                       vec_rows_lds<DT>(W, int64_t(L) * (16 / int(sizeof(DT)))), s, a, R, word_flags);
}

// Launches the row kernel for a call of F features per step if it fits one (F a multiple of
// the vector width with a power-of-two number of vectors up to 64, a row's steps within 16
// waves whose LDS fits one CU, at least kVecRowsMinGroups workgroups; x and z 16-byte aligned,
// checked by the caller) and returns whether it did. W is the fewest waves (a power of two)
// that hold a row, and a workgroup takes R = W * (steps per wave) / T whole rows.
template <typename DT, bool TR>
bool vec_rows_launch(const Args& a, int64_t F, int word_flags, hipStream_t s) {
    constexpr int V = 16 / int(sizeof(DT));
    if (F % V != 0) return false;
    const int64_t L = F / V;
    if (L > kWave || (L & (L - 1)) != 0) return false;
    const int64_t per_wave = (kWave / L) * kVecSteps;
    int W = 1;
    while (W < 16 && int64_t(W) * per_wave < a.T) W *= 2;
    if (int64_t(W) * per_wave < a.T || vec_rows_lds<DT>(W, F) > kVecRowsMaxLds) return false;
    const int R = int(int64_t(W) * per_wave / a.T);
    const int64_t groups = (a.N + R - 1) / R;
    if (groups < kVecRowsMinGroups || groups > INT32_MAX) return false;
    switch (L) {
        case 1: vec_rows_launch_l<DT, TR, 1>(a, groups, W, R, word_flags, s); break;
        case 2: vec_rows_launch_l<DT, TR, 2>(a, groups, W, R, word_flags, s); break;
        case 4: vec_rows_launch_l<DT, TR, 4>(a, groups, W, R, word_flags, s); break;
        case 8: vec_rows_launch_l<DT, TR, 8>(a, groups, W, R, word_flags, s); break;
        case 16: vec_rows_launch_l<DT, TR, 16>(a, groups, W, R, word_flags, s); break;
        case 32: vec_rows_launch_l<DT, TR, 32>(a, groups, W, R, word_flags, s); break;
        default: vec_rows_launch_l<DT, TR, 64>(a, groups, W, R, word_flags, s); break;
    }
    return true;
}

}  // namespace host
}  // namespace rlcs
