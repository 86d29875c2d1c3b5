// Block-local causal attention (Sec. 3.3, 3.6) for heads of 16 or 32
// dimensions, the head width of the paper's own model (d_model = 128, 8
// heads, Sec. 4).  At such widths a head's score is a 16- or 32-term dot
// product and the layer's cost sits in its D x D projections, so these
// kernels use plain float32 vector arithmetic: one thread per query (per key
// in the dK / dV pass), the other operand's rows staged through LDS in
// chunks of kSmChunk tokens and read by broadcast, softmax in base 2 with a
// running maximum.  The interface is that of the 64-dim two-pass path:
//   forward  out [B, T, D] at columns h*dh..; lse [B, H, T] (base 2, of the
//            scores scaled by log2(e) / sqrt(dh));
//   dq pass  dq into dqkv, delta [B, H, T] = dO . O per query;
//   dkdv     dk, dv into dqkv.
// qkv and dqkv are [B, T, 3D] with Q | K | V, head h at columns h*dh.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include "common.h"
#include "kernels.h"

namespace bcmt {
namespace {

constexpr int kSmChunk = 64;

// Rows r0 .. r0+n-1 (n <= kSmChunk) of a [*, 3D]-strided head slice (DH
// values from column `col`) into LDS as float32, zeros past n.
template <typename T, int DH>
__device__ __forceinline__ void stage_rows(float (*dst)[DH], const T* __restrict__ base, int64_t ld,
                                           int col, int r0, int n) {
  constexpr int VE = Vec16<T>::N;
  constexpr int VPR = DH / VE;  // 16-byte vectors per row
  for (int e = threadIdx.x; e < kSmChunk * VPR; e += blockDim.x) {
    const int r = e / VPR, v = e % VPR;
    typename Vec16<T>::type x{};
    if (r < n) x = load16(base + (int64_t)(r0 + r) * ld + col + v * VE);
#pragma unroll
    for (int q = 0; q < VE; ++q) dst[r][v * VE + q] = to_f32(x[q]);
  }
}

template <typename T, int DH>
__device__ __forceinline__ void load_row(float (&dst)[DH], const T* __restrict__ p) {
  constexpr int VE = Vec16<T>::N;
#pragma unroll
  for (int v = 0; v < DH / VE; ++v) {
    const auto x = load16(p + v * VE);
#pragma unroll
    for (int q = 0; q < VE; ++q) dst[v * VE + q] = to_f32(x[q]);
  }
}

template <typename T, int DH>
__device__ __forceinline__ void store_row(T* __restrict__ p, const float (&src)[DH], float scale) {
#pragma unroll
  for (int v = 0; v < DH; v += 4)
    store4(p + v, src[v] * scale, src[v + 1] * scale, src[v + 2] * scale, src[v + 3] * scale);
}

// Workgroup = (query tile of blockDim.x, block i, b * H + h).
template <typename T, int DH>
__global__ __launch_bounds__(256) void attn_small_fwd_kernel(const T* __restrict__ qkv,
                                                             T* __restrict__ out,
                                                             float* __restrict__ lse, int Tn, int D,
                                                             int H, int L, float sl2) {
  __shared__ float ks[kSmChunk][DH], vs[kSmChunk][DH];
  const int bh = blockIdx.z, b = bh / H, h = bh % H;
  const int bs = blockIdx.y * L, be = min(bs + L, Tn);
  const int t = bs + blockIdx.x * blockDim.x + threadIdx.x;
  const bool act = t < be;
  const int qend = min(bs + (int)((blockIdx.x + 1) * blockDim.x), be);  // keys [bs, qend)
  const int64_t ld = 3 * (int64_t)D;
  const T* base = qkv + (int64_t)b * Tn * ld;
  float q[DH], acc[DH];
  if (act) load_row<T, DH>(q, base + (int64_t)t * ld + h * DH);
#pragma unroll
  for (int d = 0; d < DH; ++d) {
    q[d] = act ? q[d] * sl2 : 0.f;
    acc[d] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int c0 = bs; c0 < qend; c0 += kSmChunk) {
    const int n = min(kSmChunk, qend - c0);
    __syncthreads();
    stage_rows<T, DH>(ks, base, ld, D + h * DH, c0, n);
    stage_rows<T, DH>(vs, base, ld, 2 * D + h * DH, c0, n);
    __syncthreads();
    if (act) {
      const int jn = min(n, t - c0 + 1);  // keys of this chunk at or before t
      for (int j = 0; j < jn; ++j) {
        float s = 0.f;
#pragma unroll
        for (int d = 0; d < DH; ++d) s += q[d] * ks[j][d];
        if (s > m) {  // new running maximum: rescale what was summed so far
          const float r = exp2f(m - s);
          l *= r;
#pragma unroll
          for (int d = 0; d < DH; ++d) acc[d] *= r;
          m = s;
        }
        const float p = exp2f(s - m);
        l += p;
#pragma unroll
        for (int d = 0; d < DH; ++d) acc[d] += p * vs[j][d];
      }
    }
  }
  if (act) {
    store_row<T, DH>(out + ((int64_t)b * Tn + t) * D + h * DH, acc, 1.f / l);
    lse[(int64_t)bh * Tn + t] = m + log2f(l);
  }
}

// dQ pass: thread = query t.  delta_t = dO_t . O_t;  for keys j <= t:
// p = 2^(s2 - lse), dp = dO_t . v_j, ds = p (dp - delta_t), dq += ds k_j;
// dq is scaled by 1/sqrt(dh) at the end.
template <typename T, int DH>
__global__ __launch_bounds__(256) void attn_small_dq_kernel(
    const T* __restrict__ qkv, const T* __restrict__ o, const T* __restrict__ dout,
    const float* __restrict__ lse, float* __restrict__ delta, T* __restrict__ dqkv, int Tn, int D,
    int H, int L, float sl2, float scale) {
  __shared__ float ks[kSmChunk][DH], vs[kSmChunk][DH];
  const int bh = blockIdx.z, b = bh / H, h = bh % H;
  const int bs = blockIdx.y * L, be = min(bs + L, Tn);
  const int t = bs + blockIdx.x * blockDim.x + threadIdx.x;
  const bool act = t < be;
  const int qend = min(bs + (int)((blockIdx.x + 1) * blockDim.x), be);
  const int64_t ld = 3 * (int64_t)D;
  const T* base = qkv + (int64_t)b * Tn * ld;
  float q[DH], g[DH], dq[DH];
  float lt = 0.f, dl = 0.f;
  if (act) {
    float ov[DH];
    load_row<T, DH>(q, base + (int64_t)t * ld + h * DH);
    load_row<T, DH>(g, dout + ((int64_t)b * Tn + t) * D + h * DH);
    load_row<T, DH>(ov, o + ((int64_t)b * Tn + t) * D + h * DH);
#pragma unroll
    for (int d = 0; d < DH; ++d) dl += g[d] * ov[d];
    lt = lse[(int64_t)bh * Tn + t];
    delta[(int64_t)bh * Tn + t] = dl;
  }
#pragma unroll
  for (int d = 0; d < DH; ++d) {
    q[d] = act ? q[d] * sl2 : 0.f;
    g[d] = act ? g[d] : 0.f;
    dq[d] = 0.f;
  }
  for (int c0 = bs; c0 < qend; c0 += kSmChunk) {
    const int n = min(kSmChunk, qend - c0);
    __syncthreads();
    stage_rows<T, DH>(ks, base, ld, D + h * DH, c0, n);
    stage_rows<T, DH>(vs, base, ld, 2 * D + h * DH, c0, n);
    __syncthreads();
    if (act) {
      const int jn = min(n, t - c0 + 1);
      for (int j = 0; j < jn; ++j) {
        float s = 0.f, dp = 0.f;
#pragma unroll
        for (int d = 0; d < DH; ++d) {
          s += q[d] * ks[j][d];
          dp += g[d] * vs[j][d];
        }
        const float ds = exp2f(s - lt) * (dp - dl);
#pragma unroll
        for (int d = 0; d < DH; ++d) dq[d] += ds * ks[j][d];
      }
    }
  }
  if (act) store_row<T, DH>(dqkv + ((int64_t)b * Tn + t) * ld + h * DH, dq, scale);
}

// dK / dV pass: thread = key j.  For queries t >= j of the block:
// p = 2^(s2 - lse_t), dv += p dO_t, ds = p (dO_t . v_j - delta_t),
// dk += ds q_t; dk is scaled by 1/sqrt(dh) at the end.  The queries' q, dO,
// lse and delta are staged through LDS.
template <typename T, int DH>
__global__ __launch_bounds__(256) void attn_small_dkdv_kernel(
    const T* __restrict__ qkv, const T* __restrict__ dout, const float* __restrict__ lse,
    const float* __restrict__ delta, T* __restrict__ dqkv, int Tn, int D, int H, int L, float sl2,
    float scale) {
  __shared__ float qs[kSmChunk][DH], gs[kSmChunk][DH], ls[kSmChunk], dls[kSmChunk];
  const int bh = blockIdx.z, b = bh / H, h = bh % H;
  const int bs = blockIdx.y * L, be = min(bs + L, Tn);
  const int k0 = bs + blockIdx.x * blockDim.x;
  const int j = k0 + threadIdx.x;
  const bool act = j < be;
  const int64_t ld = 3 * (int64_t)D;
  const T* base = qkv + (int64_t)b * Tn * ld;
  float kv[DH], vv[DH], dk[DH], dv[DH];
  if (act) {
    load_row<T, DH>(kv, base + (int64_t)j * ld + D + h * DH);
    load_row<T, DH>(vv, base + (int64_t)j * ld + 2 * D + h * DH);
  }
#pragma unroll
  for (int d = 0; d < DH; ++d) {
    kv[d] = act ? kv[d] * sl2 : 0.f;
    vv[d] = act ? vv[d] : 0.f;
    dk[d] = 0.f;
    dv[d] = 0.f;
  }
  for (int c0 = k0; c0 < be; c0 += kSmChunk) {  // queries from the tile's first key on
    const int n = min(kSmChunk, be - c0);
    __syncthreads();
    stage_rows<T, DH>(qs, base, ld, h * DH, c0, n);
    stage_rows<T, DH>(gs, dout + (int64_t)b * Tn * D, D, h * DH, c0, n);
    for (int e = threadIdx.x; e < kSmChunk; e += blockDim.x) {
      ls[e] = e < n ? lse[(int64_t)bh * Tn + c0 + e] : 0.f;
      dls[e] = e < n ? delta[(int64_t)bh * Tn + c0 + e] : 0.f;
    }
    __syncthreads();
    if (act) {
      for (int i = max(0, j - c0); i < n; ++i) {  // queries t = c0 + i >= j
        float s = 0.f, dp = 0.f;
#pragma unroll
        for (int d = 0; d < DH; ++d) {
          s += qs[i][d] * kv[d];
          dp += gs[i][d] * vv[d];
        }
        const float p = exp2f(s - ls[i]);
        const float ds = p * (dp - dls[i]);
#pragma unroll
        for (int d = 0; d < DH; ++d) {
          dv[d] += p * gs[i][d];
          dk[d] += ds * qs[i][d];
        }
      }
    }
  }
  if (act) {
    T* row = dqkv + ((int64_t)b * Tn + j) * ld;
    store_row<T, DH>(row + D + h * DH, dk, scale);
    store_row<T, DH>(row + 2 * D + h * DH, dv, 1.f);
  }
}

// Threads per workgroup: the block's length rounded up to whole waves, at
// most 256.
int small_threads(int lb) {
  int t = (lb + 63) / 64 * 64;
  return t > 256 ? 256 : t;
}

template <typename T, int DH>
hipError_t small_launch(int pass, const void* qkv, const void* o, const void* dout, void* out,
                        float* lse, float* delta, int B, int Tn, int D, int H, int L,
                        hipStream_t s) {
  const int lb = L < Tn ? L : Tn;
  const int nt = small_threads(lb);
  const dim3 grid((lb + nt - 1) / nt, (Tn + L - 1) / L, B * H);
  const float scale = 1.0f / sqrtf((float)DH);
  const float sl2 = 1.4426950408889634f * scale;
  if (pass == 0)
    hipLaunchKernelGGL((attn_small_fwd_kernel<T, DH>), grid, dim3(nt), 0, s, (const T*)qkv,
                       (T*)out, lse, Tn, D, H, L, sl2);
  else if (pass == 1)
    hipLaunchKernelGGL((attn_small_dq_kernel<T, DH>), grid, dim3(nt), 0, s, (const T*)qkv,
                       (const T*)o, (const T*)dout, (const float*)lse, delta, (T*)out, Tn, D, H, L,
                       sl2, scale);
  else
    hipLaunchKernelGGL((attn_small_dkdv_kernel<T, DH>), grid, dim3(nt), 0, s, (const T*)qkv,
                       (const T*)dout, (const float*)lse, (const float*)delta, (T*)out, Tn, D, H,
                       L, sl2, scale);
  return hipGetLastError();
}

template <typename T>
hipError_t small_dispatch(int pass, const void* qkv, const void* o, const void* dout, void* out,
                          float* lse, float* delta, int B, int Tn, int D, int H, int L,
                          hipStream_t s) {
  if (D / H == 16)
    return small_launch<T, 16>(pass, qkv, o, dout, out, lse, delta, B, Tn, D, H, L, s);
  if (D / H == 32)
    return small_launch<T, 32>(pass, qkv, o, dout, out, lse, delta, B, Tn, D, H, L, s);
  return hipErrorInvalidValue;
}

}  // namespace

bool attn_small_heads(int D, int H) { return D / H == 16 || D / H == 32; }

hipError_t attn_small_fwd(DType dt, const void* qkv, void* out, float* lse, int B, int T, int D,
                          int H, int L, hipStream_t s) {
  if (dt == DType::BF16)
    return small_dispatch<bf16>(0, qkv, nullptr, nullptr, out, lse, nullptr, B, T, D, H, L, s);
  return small_dispatch<float>(0, qkv, nullptr, nullptr, out, lse, nullptr, B, T, D, H, L, s);
}

hipError_t attn_small_dq(DType dt, const void* qkv, const void* o, const void* dout,
                         const float* lse, float* delta, void* dqkv, int B, int T, int D, int H,
                         int L, hipStream_t s) {
  if (dt == DType::BF16)
    return small_dispatch<bf16>(1, qkv, o, dout, dqkv, const_cast<float*>(lse), delta, B, T, D, H,
                                L, s);
  return small_dispatch<float>(1, qkv, o, dout, dqkv, const_cast<float*>(lse), delta, B, T, D, H,
                               L, s);
}

hipError_t attn_small_dkdv(DType dt, const void* qkv, const void* dout, const float* lse,
                           const float* delta, void* dqkv, int B, int T, int D, int H, int L,
                           hipStream_t s) {
  if (dt == DType::BF16)
    return small_dispatch<bf16>(2, qkv, nullptr, dout, dqkv, const_cast<float*>(lse),
                                const_cast<float*>(delta), B, T, D, H, L, s);
  return small_dispatch<float>(2, qkv, nullptr, dout, dqkv, const_cast<float*>(lse),
                               const_cast<float*>(delta), B, T, D, H, L, s);
}

}  // namespace bcmt
