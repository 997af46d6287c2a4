// wf_device.h -- device-side building blocks shared by the libwf kernels
// (gfx950 / CDNA4, wave64).  Internal header; not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wf {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;

// ---- bf16 <-> fp32 -------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(((uint32_t)b) << 16);
}

// fp32 -> bf16, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    return __builtin_bit_cast(uint16_t, (__bf16)f);
}

// Two fp32 -> one dword of two bf16 (lo in bits 0..15), one instruction.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    bf16x2 v;
    v.x = (__bf16)lo;
    v.y = (__bf16)hi;
    return __builtin_bit_cast(uint32_t, v);
}

// 2^x with the bare hardware instruction (no range reduction; results
// below the normal range flush towards zero, which softmax weights allow).
__device__ __forceinline__ float fast_exp2(float x) {
    return __builtin_amdgcn_exp2f(x);
}

// 16-byte global load reinterpreted as an MFMA bf16x8 operand.
__device__ __forceinline__ bf16x8 load_bf16x8(const uint16_t *p) {
    u32x4 v = *reinterpret_cast<const u32x4 *>(p);
    return __builtin_bit_cast(bf16x8, v);
}

// The same load with the non-temporal hint, for operands a launch reads
// exactly once (weights streamed through one workgroup): streamed at the
// caches' lowest priority they do not displace reused data (the verify
// step's LM head: 214 -> 200 us).  (The KV-only prefill keeps plain loads:
// the hint gained 14 us at the 8B shapes and lost 24 at the 32B shapes.)
__device__ __forceinline__ bf16x8 load_bf16x8_nt(const uint16_t *p) {
    u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
    return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ bf16x8 zero_bf16x8() {
    u32x4 z = {0u, 0u, 0u, 0u};
    return __builtin_bit_cast(bf16x8, z);
}

// D(16x16, fp32) += A(16x32) * B(32x16), bf16 inputs.  Lane l supplies row
// l%16 of A and column l%16 of B, eight consecutive K elements each from
// K-group l/16; it receives D rows 4*(l/16)..+3 of column l%16.  Any fixed
// assignment of K indices to (K-group, element) works as long as A and B
// use the same one.
__device__ __forceinline__ f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// ---- wavefront reductions --------------------------------------------------
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        v = fmaxf(v, __shfl_xor(v, off, kWave));
    return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        v += __shfl_xor(v, off, kWave);
    return v;
}

// ---- mergeable softmax row state -------------------------------------------
// Summary of a set T of logits z_v relative to its maximum m:
//   m  = max z,  a = lowest index attaining m,
//   sp = sum_{v in T, v != a} exp(z_v - m),
//   t  = sum_{v in T} exp(z_v - m) (z_v - m).
// Then softmax entropy over T is log1p(sp) - t / (1 + sp) (both terms >= 0,
// so a peaked row loses nothing to cancellation).  Merging is commutative
// and associative up to fp32 rounding; the argmax part is exact.
struct RowState {
    float m;
    int32_t a;
    float sp;
    float t;
};

__device__ __forceinline__ RowState state_empty() {
    RowState s;
    s.m = -INFINITY;
    s.a = 0x7fffffff;
    s.sp = 0.f;
    s.t = 0.f;
    return s;
}

__device__ __forceinline__ RowState state_single(float z, int32_t idx) {
    RowState s;
    s.m = z;
    s.a = idx;
    s.sp = 0.f;
    s.t = 0.f;
    return s;
}

__device__ __forceinline__ RowState state_merge(RowState x, RowState y) {
    // primary = larger max, lower index on a tie
    const bool swap = (y.m > x.m) || (y.m == x.m && y.a < x.a);
    RowState p = swap ? y : x;
    RowState q = swap ? x : y;
    if (q.m == -INFINITY)             // q holds only zero-probability terms
        return p;
    const float dm = q.m - p.m;       // <= 0
    const float e = expf(dm);
    const float wq = 1.f + q.sp;      // q's mass relative to its own max
    p.sp = p.sp + wq * e;
    p.t = p.t + e * (q.t + wq * dm);
    return p;
}

__device__ __forceinline__ RowState shfl_xor_state(RowState s, int off) {
    RowState o;
    o.m = __shfl_xor(s.m, off, kWave);
    o.a = __shfl_xor(s.a, off, kWave);
    o.sp = __shfl_xor(s.sp, off, kWave);
    o.t = __shfl_xor(s.t, off, kWave);
    return o;
}

// Butterfly merge across the wave; every lane ends with the same state.
__device__ __forceinline__ RowState wave_merge(RowState s) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        s = state_merge(s, shfl_xor_state(s, off));
    return s;
}

__device__ __forceinline__ float state_entropy(RowState s) {
    return log1pf(s.sp) - s.t / (1.f + s.sp);
}

// Index of the calling wave in its workgroup, as a wave-uniform (scalar)
// value: derived from threadIdx.x the compiler would treat it as varying per
// lane and turn every branch on it into a divergent one.
__device__ __forceinline__ int wave_id() {
    return __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
}

// Halves of a device-scope fence.
__device__ __forceinline__ void fence_release_agent() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
}
__device__ __forceinline__ void fence_acquire_agent() {
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
}

// "Last workgroup to arrive finishes the reduction": every workgroup calls
// this once its results are stored; it returns true (uniformly within the
// workgroup) in the one workgroup that draws the last of `expected` tickets
// from *counter, and that workgroup then sees every other workgroup's stored
// results.  The workgroup barrier orders all threads' stores before thread
// 0's device-scope release, so the L2 write-back runs once per workgroup,
// and only the last workgroup pays for the acquire.  The caller resets the
// counter to zero when it is done.
__device__ __forceinline__ bool arrive_last(unsigned *counter, unsigned expected) {
    __shared__ int last;
    __syncthreads();
    if (threadIdx.x == 0) {
        fence_release_agent();
        const bool l = atomicAdd(counter, 1u) == expected - 1u;
        if (l)
            fence_acquire_agent();
        last = l;
    }
    __syncthreads();
    return last != 0;
}

}  // namespace wf
