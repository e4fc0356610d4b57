// Device helpers shared by the decode kernels (kernels.hip) and the prefill
// kernel (prefill.hip), gfx950 only.
#pragma once

#include <hip/hip_runtime.h>

#include <cfloat>
#include <cstdint>

namespace ca {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

typedef __fp16 fp16x4_t __attribute__((__vector_size__(4 * sizeof(__fp16))));

// ds_read_b64_tr_b16: each lane names 4 consecutive halves in LDS; within
// every 16-lane group, lane i receives element i % 4 of the values named by
// lanes 4j + i / 4, for j = 0..3. With lane (i, group g) naming row
// r0 + 4g + i / 4, column c0 + 4 (i % 4) of a row-major [row][col] tile,
// lane i gets rows r0 + 4g + j, column c0 + i: the 16x16x16 MFMA A operand
// of the transposed tile, without a transposed copy.
__device__ __forceinline__ half4 lds_read_tr16(const _Float16* p) {
  const fp16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4f16(
      (__attribute__((address_space(3))) fp16x4_t*)(p));
  return __builtin_bit_cast(half4, v);
}

constexpr float kNegBig = -FLT_MAX;  // "no score yet": exp2(kNegBig - x) == 0, never NaN

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, true));
}

// Sum over aligned groups of N lanes (N = 8, 16, 32 or 64); every lane of the
// group receives the sum. Must be called with the whole wavefront active.
template <int N>
__device__ __forceinline__ float group_sum(float x) {
  x += dpp<0xB1>(x);   // quad_perm [1,0,3,2]
  x += dpp<0x4E>(x);   // quad_perm [2,3,0,1]
  x += dpp<0x141>(x);  // row_half_mirror: groups of 8
  if constexpr (N >= 16) x += dpp<0x140>(x);  // row_mirror: rows of 16
  if constexpr (N >= 32) x += __shfl_xor(x, 16);
  if constexpr (N >= 64) x += __shfl_xor(x, 32);
  return x;
}

// Maximum over the four 16-lane rows of a wavefront (lanes l, l^16, l^32,
// l^48) with gfx950's row-swap moves instead of LDS permutes. Swapping a
// register with a copy of itself, odd rows against even rows, leaves rows
// 2k and 2k+1 of the value in the two registers of every lane of both rows;
// the half swap does the same for the two 32-lane halves. The s_nop covers
// the wait states the swap needs after a vector write of its operands.
__device__ __forceinline__ void swap_rows16(float& a, float& b) {
  asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}
__device__ __forceinline__ void swap_halves32(float& a, float& b) {
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}
__device__ __forceinline__ float rows4_max(float x) {
  float a = x, b = x;
  swap_rows16(a, b);
  float c = fmaxf(a, b), d = c;
  swap_halves32(c, d);
  return fmaxf(c, d);
}

template <typename T>
struct Elem;
template <>
struct Elem<_Float16> {
  static constexpr int kPerVec = 8;  // elements per 16-byte vector
  __device__ static __forceinline__ void unpack(const uint4& r, float* f) {
    const half8 h = __builtin_bit_cast(half8, r);
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = static_cast<float>(h[i]);
  }
  __device__ static __forceinline__ uint4 pack(const float* f) {
    half8 h;
#pragma unroll
    for (int i = 0; i < 8; ++i) h[i] = static_cast<_Float16>(f[i]);
    return __builtin_bit_cast(uint4, h);
  }
};
template <>
struct Elem<float> {
  static constexpr int kPerVec = 4;
  __device__ static __forceinline__ void unpack(const uint4& r, float* f) {
    f[0] = __uint_as_float(r.x);
    f[1] = __uint_as_float(r.y);
    f[2] = __uint_as_float(r.z);
    f[3] = __uint_as_float(r.w);
  }
  __device__ static __forceinline__ uint4 pack(const float* f) {
    return make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]),
                      __float_as_uint(f[3]));
  }
};

// attn_reduce (Eqn 2) in base 2: fold (mo, no, acco) into (m, n, acc).
template <int E>
__device__ __forceinline__ void fold(float& m, float& n, float* acc, float mo, float no,
                                     const float* acco) {
  const float mm = fmaxf(m, mo);
  const float a = fast_exp2(m - mm);
  const float b = fast_exp2(mo - mm);
  n = n * a + no * b;
#pragma unroll
  for (int j = 0; j < E; ++j) acc[j] = acc[j] * a + acco[j] * b;
  m = mm;
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x = fmaxf(x, __shfl_xor(x, off));
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

__device__ __forceinline__ float readlane_f(float x, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Compiler-only barrier: emits no instruction, but no memory access is moved
// across it (it pins the program order the exchange below relies on).
__device__ __forceinline__ void compiler_fence() { __atomic_signal_fence(__ATOMIC_SEQ_CST); }

// vmcnt(0): every vector memory access this wavefront issued before the call
// has completed (for a device-scope store: it is visible to every XCD).
__device__ __forceinline__ void wait_stores() {
  compiler_fence();
  __builtin_amdgcn_s_waitcnt(0x0F70);
  compiler_fence();
}

// Exchange of partial results between blocks of one launch (the blocks may
// sit on different XCDs, whose L2 caches are not coherent with each other).
// The HIP memory model would express it as a release fetch_add by each
// writer and an acquire by the last one; at agent scope that costs a whole
// L2 writeback and invalidate per block (measured 2.5x slower on the decode
// call). The protocol below gets the same ordering per access instead:
//  1. Writers store their part only with device-scope accesses (st_dev,
//     st_dev4: the sc1 bit), which write through the XCD's L2, so a
//     completed store is visible to loads from any XCD; nothing else the
//     reader needs is stored by the writer.
//  2. Every wavefront that stored waits for its stores to complete
//     (wait_stores: s_waitcnt vmcnt(0)), and the block meets at a barrier
//     (when more than one wavefront stored) before one thread counts the
//     arrival with an atomic add at device scope (arrive_last). So the
//     count is performed only after the whole part is visible.
//  3. The thread whose add returns need - 1 is last: every other part was
//     visible before its writer counted. The reader branches on that value
//     before issuing any load of the parts (the hardware does not issue
//     loads speculatively past a branch), and it reads them only with
//     device-scope loads (ld_dev, ld_dev4: sc1), which do not return stale
//     lines of its own L1 or L2.
//  4. compiler_fence() in wait_stores and arrive_last keeps the compiler
//     from sinking a part store below the wait or the count, or hoisting a
//     part load above the count. Moving any part access across those
//     points, or reading a part with an ordinary (non-sc1) load, breaks the
//     protocol.
// The last contributor also resets the counter to 0, so counters are zero
// between launches (the next launch is ordered after it by the stream).
__device__ __forceinline__ void st_dev(float* p, float x) {
  __hip_atomic_store(p, x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_dev(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ bool arrive_last(int32_t* c, int need) {
  compiler_fence();
  const int old = __hip_atomic_fetch_add(c, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (old != need - 1) return false;
  compiler_fence();
  __hip_atomic_store(c, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return true;
}

// Partial O vectors move as 16-byte raw buffer accesses with the sc1 bit
// (device scope; the exchange protocol above) over the partial-O workspace
// (descriptor word 3 is the gfx9 raw-buffer format; byte offsets are
// 32-bit, the host keeps that region below 4 GiB).
constexpr int kRsrcWord3 = 0x00020000;
constexpr int kDevScope = 16;  // cache-policy bit sc1
__device__ __forceinline__ __amdgpu_buffer_rsrc_t part_rsrc(const float* ws_o, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(ws_o), 0, static_cast<int>(bytes),
                                           kRsrcWord3);
}
__device__ __forceinline__ float4 ld_dev4(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, static_cast<int>(off), 0, kDevScope);
  return make_float4(__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z),
                     __uint_as_float(v.w));
}
__device__ __forceinline__ void st_dev4(__amdgpu_buffer_rsrc_t r, uint32_t off, float a, float b,
                                        float c, float d) {
  const u32x4 v = {__float_as_uint(a), __float_as_uint(b), __float_as_uint(c), __float_as_uint(d)};
  __builtin_amdgcn_raw_buffer_store_b128(v, r, static_cast<int>(off), 0, kDevScope);
}

}  // namespace
}  // namespace ca
