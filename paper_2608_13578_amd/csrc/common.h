// Device-side building blocks shared by the BCMT kernels (gfx950 / CDNA4).
//
// Element types: the layer runs either in float32 end to end or with
// bfloat16 storage and float32 accumulation.  Matrix products use the CDNA4
// matrix cores through two instruction shapes that share one register
// layout:
//   bf16: v_mfma_f32_16x16x32_bf16  (one instruction per 32-wide K step)
//   f32 : v_mfma_f32_16x16x4_f32    (eight instructions per 32-wide K step)
// For both, lane l of a wave supplies, for row/column (l % 16), the eight
// consecutive K elements 8*(l/16) .. 8*(l/16)+7 of a 32-wide K step.  For
// f32 the eight instructions j = 0..7 each contract the elements j of the
// four lane groups; together they cover the same 32 K values (the order of
// the K summation differs, nothing else).
// The 16x16 float32 result lands with lane l holding column (l % 16) and
// rows 4*(l/16) .. 4*(l/16)+3.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bcmt {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));

constexpr int kWave = 64;

template <typename T> struct Frag;
template <> struct Frag<bf16> { typedef bf16x8 type; };
template <> struct Frag<float> { typedef f32x8 type; };

// acc += A_frag (16 x 32) * B_frag (32 x 16), operands in the layout above.
__device__ __forceinline__ f32x4 mma16(const bf16x8& a, const bf16x8& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma16(const f32x8& a, const f32x8& b, f32x4 c) {
#pragma unroll
  for (int j = 0; j < 8; ++j) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], b[j], c, 0, 0, 0);
  return c;
}

// Scalar conversions.
__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }
template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }

// 16-byte vectors: 8 bf16 or 4 float.
template <typename T> struct Vec16;
template <> struct Vec16<bf16> {
  static constexpr int N = 8;
  typedef bf16x8 type;
};
template <> struct Vec16<float> {
  static constexpr int N = 4;
  typedef f32x4 type;
};

template <typename T>
__device__ __forceinline__ typename Vec16<T>::type load16(const T* p) {
  return *reinterpret_cast<const typename Vec16<T>::type*>(p);
}
template <typename T>
__device__ __forceinline__ void store16(T* p, const typename Vec16<T>::type& v) {
  *reinterpret_cast<typename Vec16<T>::type*>(p) = v;
}

// Store four consecutive values converted to T (8 bytes for bf16, 16 for f32).
__device__ __forceinline__ void store4(float* p, float a, float b, float c, float d) {
  f32x4 v = {a, b, c, d};
  *reinterpret_cast<f32x4*>(p) = v;
}
__device__ __forceinline__ void store4(bf16* p, float a, float b, float c, float d) {
  bf16x4 v = {(bf16)a, (bf16)b, (bf16)c, (bf16)d};
  *reinterpret_cast<bf16x4*>(p) = v;
}
// Load four consecutive values as float.
__device__ __forceinline__ f32x4 load4f(const float* p) { return *reinterpret_cast<const f32x4*>(p); }
__device__ __forceinline__ f32x4 load4f(const bf16* p) {
  bf16x4 v = *reinterpret_cast<const bf16x4*>(p);
  f32x4 r = {(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
  return r;
}

// The gate G = sigmoid(U), kept for the backward pass, is stored as fp16
// when the layer runs in bf16: the same two bytes, eight times finer
// steps on (0, 1).  Its block sums of dY * G feed the memory's and the
// decay's gradients, which cancel heavily.
typedef _Float16 f16;
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
template <typename T> struct GateT { typedef T type; };
template <> struct GateT<bf16> { typedef f16 type; };
__device__ __forceinline__ float to_f32(f16 x) { return (float)x; }
__device__ __forceinline__ void store4(f16* p, float a, float b, float c, float d) {
  f16x4 v = {(f16)a, (f16)b, (f16)c, (f16)d};
  *reinterpret_cast<f16x4*>(p) = v;
}

// Wave-wide reductions over all 64 lanes.
// Wave-wide sum / max, returned to every lane; the whole wave must be
// active.  Within each row of 16 lanes, DPP moves (xor 1 and xor 2 inside
// quads, then the half-row and row mirrors) combine values without the LDS
// crossbar; the four row results are then read into scalar registers.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                               0xF, 0xF, false));
}
__device__ __forceinline__ float lane_f(float v, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_mov<0xB1>(v);   // quad_perm [1, 0, 3, 2]
  v += dpp_mov<0x4E>(v);   // quad_perm [2, 3, 0, 1]
  v += dpp_mov<0x141>(v);  // row_half_mirror
  v += dpp_mov<0x140>(v);  // row_mirror
  return (lane_f(v, 0) + lane_f(v, 16)) + (lane_f(v, 32) + lane_f(v, 48));
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_mov<0xB1>(v));
  v = fmaxf(v, dpp_mov<0x4E>(v));
  v = fmaxf(v, dpp_mov<0x141>(v));
  v = fmaxf(v, dpp_mov<0x140>(v));
  return fmaxf(fmaxf(lane_f(v, 0), lane_f(v, 16)), fmaxf(lane_f(v, 32), lane_f(v, 48)));
}

__device__ __forceinline__ float sigmoidf_(float u) {
  // 1 / (1 + e^-u) for u >= 0 and e^u / (1 + e^u) for u < 0: both forms only
  // ever exponentiate -|u|, so neither overflows nor cancels.
  float e = __expf(-fabsf(u));
  float r = 1.0f / (1.0f + e);
  return u >= 0.0f ? r : e * r;
}

// Fragment loads from LDS: 8 consecutive elements (16 bytes for bf16, 32 for
// f32; the f32 case is read as two 16-byte halves so that only 16-byte
// alignment is needed).
__device__ __forceinline__ bf16x8 load_frag(const bf16* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}
__device__ __forceinline__ f32x8 load_frag(const float* p) {
  f32x4 lo = *reinterpret_cast<const f32x4*>(p);
  f32x4 hi = *reinterpret_cast<const f32x4*>(p + 4);
  f32x8 r = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return r;
}
// Fragment made of two runs of four consecutive elements (p[0..3], q[0..3]).
__device__ __forceinline__ bf16x8 load_frag_split(const bf16* p, const bf16* q) {
  bf16x4 a = *reinterpret_cast<const bf16x4*>(p);
  bf16x4 b = *reinterpret_cast<const bf16x4*>(q);
  bf16x8 r = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  return r;
}
__device__ __forceinline__ f32x8 load_frag_split(const float* p, const float* q) {
  f32x4 a = *reinterpret_cast<const f32x4*>(p);
  f32x4 b = *reinterpret_cast<const f32x4*>(q);
  f32x8 r = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  return r;
}
// Fragment from two f32x4 register tiles, converted to T.
template <typename T> __device__ __forceinline__ typename Frag<T>::type frag_from(const f32x4& a, const f32x4& b);
template <> __device__ __forceinline__ bf16x8 frag_from<bf16>(const f32x4& a, const f32x4& b) {
  bf16x8 r = {(bf16)a[0], (bf16)a[1], (bf16)a[2], (bf16)a[3], (bf16)b[0], (bf16)b[1], (bf16)b[2], (bf16)b[3]};
  return r;
}
template <> __device__ __forceinline__ f32x8 frag_from<float>(const f32x4& a, const f32x4& b) {
  f32x8 r = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  return r;
}

// 8 consecutive elements as float32, and back.
__device__ __forceinline__ void ld8(const bf16* p, float (&o)[8]) {
  const bf16x8 v = *reinterpret_cast<const bf16x8*>(p);
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = (float)v[e];
}
__device__ __forceinline__ void ld8(const float* p, float (&o)[8]) {
  const f32x4 a = *reinterpret_cast<const f32x4*>(p), b = *reinterpret_cast<const f32x4*>(p + 4);
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    o[e] = a[e];
    o[4 + e] = b[e];
  }
}
__device__ __forceinline__ void st8(bf16* p, const float (&v)[8]) {
  bf16x8 o;
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = (bf16)v[e];
  *reinterpret_cast<bf16x8*>(p) = o;
}
__device__ __forceinline__ void st8(f16* p, const float (&v)[8]) {
  f16x8 o;
#pragma unroll
  for (int k = 0; k < 8; ++k) o[k] = (f16)v[k];
  *reinterpret_cast<f16x8*>(p) = o;
}
__device__ __forceinline__ void st8(float* p, const float (&v)[8]) {
  *reinterpret_cast<f32x4*>(p) = f32x4{v[0], v[1], v[2], v[3]};
  *reinterpret_cast<f32x4*>(p + 4) = f32x4{v[4], v[5], v[6], v[7]};
}

// 2^x with one v_exp_f32: results below the smallest normal float flush to
// zero (exp2f adds a range reduction for them), which a softmax weight
// can afford.
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// ------------------------------------------------------------------ LDS helpers
typedef __attribute__((address_space(3))) void lds_void_t;
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4_t;

// ds_read_b64_tr_b16 through inline assembly.  The compiler's wait insertion
// assumes that the builtin form may read LDS still being written by any
// direct global->LDS load in flight and drains all of them first
// (s_waitcnt vmcnt(0)), which would also wait for the tiles being
// prefetched.  Callers order these reads after their own vmcnt wait and
// barrier for the tile they read, wait for them with lds_tr_wait() (or
// lds_wait<N>()) and pass every result through lds_tr_bind() before using
// it: the compiler does not count these reads in its LDS wait bookkeeping.
__device__ __forceinline__ bf16x4 lds_read_tr(const bf16* p) {
  s16x4 v;
  const unsigned a = (unsigned)(uintptr_t)((lds_s16x4_t*)(p));
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(v) : "v"(a));
  return __builtin_bit_cast(bf16x4, v);
}
// 16-byte LDS read in inline assembly, for data written by direct
// global->LDS loads; same contract as lds_read_tr().
__device__ __forceinline__ f32x4 lds_read_f32x4(const float* p) {
  f32x4 v;
  const unsigned a = (unsigned)(uintptr_t)((__attribute__((address_space(3))) float*)(p));
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(a));
  return v;
}
// 4-byte LDS read in inline assembly; same contract as lds_read_tr().
__device__ __forceinline__ float lds_read_f32(const float* p) {
  float v;
  const unsigned a = (unsigned)(uintptr_t)((__attribute__((address_space(3))) float*)(p));
  asm volatile("ds_read_b32 %0, %1" : "=v"(v) : "v"(a));
  return v;
}
// 16-byte bf16 LDS read in inline assembly; same contract as lds_read_tr().
__device__ __forceinline__ bf16x8 lds_read_b128(const bf16* p) {
  bf16x8 v;
  const unsigned a = (unsigned)(uintptr_t)((__attribute__((address_space(3))) bf16*)(p));
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(a));
  return v;
}
// Waits for every outstanding LDS read of this wave.
__device__ __forceinline__ void lds_tr_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
// Waits until at most N of this wave's LDS reads are outstanding (they
// complete in issue order).  Only for stretches of code whose LDS and scalar
// memory traffic is all issued through the inline-assembly reads above.
template <int N>
__device__ __forceinline__ void lds_wait() {
  static_assert(N >= 0 && N <= 15, "lgkmcnt range");
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
}
// Ties a value to the preceding lds_tr_wait(), so that no use of it is
// scheduled before the wait.
template <class V>
__device__ __forceinline__ void lds_tr_bind(V& v) {
  asm volatile("" : "+v"(v));
}

}  // namespace bcmt
