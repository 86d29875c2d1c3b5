// Incremental decoding: the layer's output for one more token of each of B
// sequences, given what the earlier tokens left in a decode state.
//
// The layer is causal (Sec. 3.6): token t of block i needs only the keys and
// values of tokens s <= t of block i (Sec. 3.3) and the context C_i, which
// depends on earlier blocks only (Sec. 3.5, 3.7).  So a step computes, per
// sequence,
//   [q k v] = x [Wq Wk Wv]            (k, v appended to the block's cache)
//   o       = softmax(q K^T / 8) V    (over the block's cached tokens)
//   h       = o Wo,  s = h . wp       (h and s appended to the block's cache)
//   y       = h + sigmoid(h Wg) * C_i (+ x)
// and after the block's last token pools the block (Sec. 3.4), advances the
// memory recurrence N = g N + S, Z = g Z + 1 (Sec. 3.5) and forms the next
// block's context C = (N / Z) Wm.
//
// The products have a handful of rows (the sequences) against a [D, N]
// weight: they are weight-streaming matrix-vector products, and what bounds
// them is how many loads are in flight per CU.  So each product is split
// into 250-400 workgroups of a few KB of weights each (64 columns x 32-128
// rows, one round of 16-byte loads per lane), writing partial sums per K
// split; a second small kernel adds the splits in a fixed order and applies
// the step's epilogue (for the QKV product the attention kernel does it).
// The kernel boundary makes the partials visible across the chip's L2s, so
// nothing synchronises inside a kernel, and every run gives the same result.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "common.h"
#include "kernels.h"

namespace bcmt {
namespace {

constexpr int kDvB = 8;                     // sequences per workgroup
constexpr int kDvLanesPerRow = 8;           // a row of the column tile: 8 lanes x 16 bytes
constexpr int kDvRowsPerWave = 64 / kDvLanesPerRow;
constexpr int kDvRowStep = 4 * kDvRowsPerWave;  // rows per round of the 4 waves (32)
constexpr int kDvMaxKc = 128;               // K rows per workgroup at most (4 rounds)
constexpr int kDecMaxBatch = 64;

template <typename T>
constexpr int dv_cols() { return kDvLanesPerRow * Vec16<T>::N; }

// The weight as up to three column segments of width seg (Wq | Wk | Wv).
template <typename T>
struct DvW {
  const T* w[3];
  int seg;
  int64_t ld;
  __device__ __forceinline__ const T* col(int n) const {
    const int s = n / seg;
    return w[s] + (n - s * seg);
  }
};

// part[ky][b][n] = sum over the rows k of split ky of x[b, k] W[k, n], for a
// column tile of CT columns, kc rows (a multiple of 32) and up to kDvB
// sequences per workgroup.  Lane (column vector cg, row lane rl) of wave w
// takes rows w*8 + rl + 32u; the row lanes meet by shuffles, the waves in
// LDS.
template <typename T>
__global__ __launch_bounds__(256) void dec_gemv_part_kernel(const T* __restrict__ x, int64_t ldx,
                                                            int B, DvW<T> w, int K, int N, int kc,
                                                            float* __restrict__ part) {
  constexpr int VE = Vec16<T>::N, CT = dv_cols<T>();
  __shared__ float xs[kDvB][kDvMaxKc];
  __shared__ float red[4][kDvB][CT];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n0 = blockIdx.x * CT;
  const int k0 = blockIdx.y * kc;
  const int b0 = blockIdx.z * kDvB;
  const int nbt = min(kDvB, B - b0);
  const int kn = min(kc, K - k0);
  // The weight tile's loads go out first; x (tiny) is staged meanwhile.
  const int cg = lane % kDvLanesPerRow, rl = lane / kDvLanesPerRow;
  const T* wcol = w.col(n0 + cg * VE) + (int64_t)k0 * w.ld;
  constexpr int U = kDvMaxKc / kDvRowStep;
  typename Vec16<T>::type wv[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int r = wave * kDvRowsPerWave + rl + u * kDvRowStep;
    wv[u] = r < kn ? load16(wcol + (int64_t)r * w.ld) : typename Vec16<T>::type{};
  }
  // x[b0.., k0..k0+kc) as 16-byte vectors (kc and K are multiples of 32).
  {
    const int kv = kc / VE;
    for (int e = tid; e < kDvB * kv; e += blockDim.x) {
      const int b = e / kv, k = (e - b * kv) * VE;
      const auto v = (b < nbt && k < kn) ? load16(x + (int64_t)(b0 + b) * ldx + k0 + k)
                                         : typename Vec16<T>::type{};
#pragma unroll
      for (int q = 0; q < VE; ++q) xs[b][k + q] = to_f32(v[q]);
    }
  }
  __syncthreads();
  float acc[kDvB][VE];
#pragma unroll
  for (int b = 0; b < kDvB; ++b)
#pragma unroll
    for (int e = 0; e < VE; ++e) acc[b][e] = 0.f;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int r = wave * kDvRowsPerWave + rl + u * kDvRowStep;
    if (r < kn) {
#pragma unroll
      for (int b = 0; b < kDvB; ++b) {
        const float xb = xs[b][r];
#pragma unroll
        for (int e = 0; e < VE; ++e) acc[b][e] += xb * to_f32(wv[u][e]);
      }
    }
  }
  // The 8 row lanes of a column vector (lane bits 3-5) reduce-scatter their
  // sums over the 8 sequences: at each step a lane keeps the half of its
  // sequences whose bit matches its own row-lane bit and receives the
  // partner's sums for them, so that row lane r ends with sequence r's sums
  // (56 shuffles per lane instead of 192, each step's shuffles independent).
  float h4[4][VE], h2[2][VE], h1[VE];
  {
    const bool p = rl & 1;
    float snd[4][VE];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < VE; ++e) snd[i][e] = p ? acc[2 * i][e] : acc[2 * i + 1][e];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < VE; ++e) snd[i][e] = __shfl_xor(snd[i][e], 8);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < VE; ++e) h4[i][e] = (p ? acc[2 * i + 1][e] : acc[2 * i][e]) + snd[i][e];
  }
  {  // h4[i] holds sequence 2i + (rl & 1)
    const bool p = (rl >> 1) & 1;
    float snd[2][VE];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int e = 0; e < VE; ++e) snd[i][e] = p ? h4[2 * i][e] : h4[2 * i + 1][e];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int e = 0; e < VE; ++e) snd[i][e] = __shfl_xor(snd[i][e], 16);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int e = 0; e < VE; ++e) h2[i][e] = (p ? h4[2 * i + 1][e] : h4[2 * i][e]) + snd[i][e];
  }
  {  // h2[i] holds sequence 4i + (rl & 3)
    const bool p = (rl >> 2) & 1;
    float snd[VE];
#pragma unroll
    for (int e = 0; e < VE; ++e) snd[e] = p ? h2[0][e] : h2[1][e];
#pragma unroll
    for (int e = 0; e < VE; ++e) snd[e] = __shfl_xor(snd[e], 32);
#pragma unroll
    for (int e = 0; e < VE; ++e) h1[e] = (p ? h2[1][e] : h2[0][e]) + snd[e];
  }
  // h1 holds sequence rl's sums for this lane's column vector
#pragma unroll
  for (int e = 0; e < VE; ++e) red[wave][rl][cg * VE + e] = h1[e];
  __syncthreads();
  for (int e = tid; e < nbt * CT; e += blockDim.x) {
    const int b = e / CT, c = e % CT;
    part[((int64_t)blockIdx.y * B + b0 + b) * N + n0 + c] =
        (red[0][b][c] + red[1][b][c]) + (red[2][b][c] + red[3][b][c]);
  }
}

// Sum of the K splits of output (b, n), in split order; eight splits' loads
// are issued before they are added.
__device__ __forceinline__ float dv_sum(const float* __restrict__ part, int ks, int B, int N, int b,
                                        int n) {
  const int64_t stride = (int64_t)B * N;
  const float* p = part + (int64_t)b * N + n;
  float v = 0.f;
  int s = 0;
  for (; s + 8 <= ks; s += 8) {
    float t[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) t[u] = p[(s + u) * stride];
#pragma unroll
    for (int u = 0; u < 8; ++u) v += t[u];
  }
  for (; s < ks; ++s) v += p[s * stride];
  return v;
}

// h = o Wo into the block cache at slot off, and per 64 columns the part of
// the pooling score h . wp.  Thread = column n of sequence blockIdx.y.
template <typename T>
__global__ __launch_bounds__(256) void dec_wo_finish_kernel(const float* __restrict__ part, int ks,
                                                            int B, int D, const T* __restrict__ wp,
                                                            T* __restrict__ Hc,
                                                            float* __restrict__ spc, int L,
                                                            int off) {
  const int b = blockIdx.y, n = blockIdx.x * blockDim.x + threadIdx.x;
  const bool on = n < D;
  const float v = on ? dv_sum(part, ks, B, D, b, n) : 0.f;
  if (on) Hc[((int64_t)b * L + off) * D + n] = from_f32<T>(v);
  const float sc = wave_sum(on ? v * to_f32(wp[n]) : 0.f);
  if ((threadIdx.x & 63) == 0 && on) spc[((int64_t)b * L + off) * (D / 64) + n / 64] = sc;
}

// y = h + sigmoid(u) C (+ x), u = h Wg.
template <typename T>
__global__ __launch_bounds__(256) void dec_gate_finish_kernel(const float* __restrict__ part,
                                                              int ks, int B, int D,
                                                              const T* __restrict__ Hc,
                                                              const float* __restrict__ C,
                                                              const T* __restrict__ x,
                                                              T* __restrict__ y, int L, int off) {
  const int b = blockIdx.y, n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= D) return;
  const float u = dv_sum(part, ks, B, D, b, n);
  const int64_t row = (int64_t)b * D + n;
  float out = to_f32(Hc[((int64_t)b * L + off) * D + n]) + sigmoidf_(u) * C[row];
  if (x) out += to_f32(x[row]);
  y[row] = from_f32<T>(out);
}

// C = Mt Wm for the next block, Z = g Z + 1 (per channel with gvec).
__global__ __launch_bounds__(256) void dec_mem_finish_kernel(const float* __restrict__ part,
                                                             int ks, int B, int D,
                                                             float* __restrict__ C,
                                                             float* __restrict__ Z, float gamma,
                                                             const float* __restrict__ gvec) {
  const int b = blockIdx.y, n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= D) return;
  const int64_t o = (int64_t)b * D + n;
  C[o] = dv_sum(part, ks, B, D, b, n);
  if (gvec) Z[o] = gvec[n] * Z[o] + 1.f;
  else if (n == 0) Z[b] = gamma * Z[b] + 1.f;
}

// Attention of the new token over the block's tokens 0..off, one workgroup
// per (head, sequence).  First the QKV product's K splits are added for
// this head: q, and the new token's k and v, which go to the block cache at
// slot off and are also kept in LDS for this token's own score and value.
// Scores: one cached key per thread (its 64 dims as 16-byte loads issued
// together).  Output: thread (16-byte vector v of the head's dims, key
// group g) adds p_j V[j] over the cached keys j = g mod G with four keys'
// loads in flight; the groups meet in LDS.
constexpr int kDecMaxL = 4096;

template <typename T>
__global__ __launch_bounds__(256) void dec_attn_kernel(const float* __restrict__ part, int ks,
                                                       int B, T* __restrict__ Kc,
                                                       T* __restrict__ Vc, T* __restrict__ o,
                                                       int D, int L, int off) {
  constexpr int VE = Vec16<T>::N, NV = 64 / VE;  // 16-byte vectors per head row
  constexpr int G = 256 / NV;                     // key groups
  __shared__ float qkv[3][64];                    // q (scaled by 1/8), k, v of the new token
  __shared__ float sc[kDecMaxL];
  __shared__ float red[G][64];
  __shared__ float wr[4];
  const int tid = threadIdx.x, h = blockIdx.x, b = blockIdx.y;
  if (tid < 192) {
    const int which = tid / 64, d = tid % 64;
    const float v = dv_sum(part, ks, B, 3 * D, b, which * D + h * 64 + d);
    const T vt = from_f32<T>(v);  // Q, K and V are stored in the compute type
    qkv[which][d] = to_f32(vt) * (which == 0 ? 0.125f : 1.f);
    if (which > 0) (which == 1 ? Kc : Vc)[((int64_t)b * L + off) * D + h * 64 + d] = vt;
  }
  __syncthreads();
  const int n = off + 1;
  float mx = -INFINITY;
  for (int j = tid; j < n; j += blockDim.x) {
    float d = 0.f;
    if (j == off) {
      for (int e = 0; e < 64; ++e) d += qkv[0][e] * qkv[1][e];
    } else {
      const T* kr = Kc + ((int64_t)b * L + j) * D + h * 64;
      typename Vec16<T>::type kv[NV];
#pragma unroll
      for (int v = 0; v < NV; ++v) kv[v] = load16(kr + v * VE);
#pragma unroll
      for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int e = 0; e < VE; ++e) d += qkv[0][v * VE + e] * to_f32(kv[v][e]);
    }
    sc[j] = d;
    mx = fmaxf(mx, d);
  }
  mx = wave_max(mx);
  if ((tid & 63) == 0) wr[tid >> 6] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(wr[0], wr[1]), fmaxf(wr[2], wr[3]));
  float sum = 0.f;
  for (int j = tid; j < n; j += blockDim.x) {
    const float p = __expf(sc[j] - mx);
    sc[j] = p;
    sum += p;
  }
  sum = wave_sum(sum);
  __syncthreads();  // wr[] reads above are done; sc[] is complete
  if ((tid & 63) == 0) wr[tid >> 6] = sum;
  __syncthreads();
  const float total = (wr[0] + wr[1]) + (wr[2] + wr[3]);
  const int vi = tid % NV, g = tid / NV;
  float acc[VE];
#pragma unroll
  for (int e = 0; e < VE; ++e) acc[e] = 0.f;
  const T* vb = Vc + (int64_t)b * L * D + h * 64 + vi * VE;
  constexpr int U = 4;
  for (int j0 = g; j0 < off; j0 += U * G) {  // the cached tokens before this one
    typename Vec16<T>::type vv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u * G;
      vv[u] = j < off ? load16(vb + (int64_t)j * D) : typename Vec16<T>::type{};
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u * G;
      const float p = j < off ? sc[j] : 0.f;
#pragma unroll
      for (int e = 0; e < VE; ++e) acc[e] += p * to_f32(vv[u][e]);
    }
  }
  if (g == off % G)  // the new token itself
#pragma unroll
    for (int e = 0; e < VE; ++e) acc[e] += sc[off] * qkv[2][vi * VE + e];
#pragma unroll
  for (int e = 0; e < VE; ++e) red[g][vi * VE + e] = acc[e];
  __syncthreads();
  if (tid < 64) {
    float t = 0.f;
    for (int k = 0; k < G; ++k) t += red[k][tid];
    o[(int64_t)b * D + h * 64 + tid] = from_f32<T>(t / total);
  }
}

// After a block's last token: a = softmax of the block's scores, S = sum_t
// a_t H[t] for 64 columns per workgroup, N = g N + S, and the new memory
// N / (g Z + 1) in the compute type (Z itself advances in the W_m product).
// Thread (16-byte vector v of the 64 columns, token group g) adds its
// tokens t = g mod G with four tokens' loads in flight.
template <typename T>
__global__ __launch_bounds__(256) void dec_pool_kernel(const T* __restrict__ Hc,
                                                       const float* __restrict__ spc, int np,
                                                       float* __restrict__ N,
                                                       const float* __restrict__ Z,
                                                       T* __restrict__ Mt, int D, int L,
                                                       float gamma,
                                                       const float* __restrict__ gvec) {
  constexpr int VE = Vec16<T>::N, NV = 64 / VE, G = 256 / NV;
  __shared__ float a[kDecMaxL];
  __shared__ float red[G][64];
  __shared__ float wr[4];
  const int tid = threadIdx.x, b = blockIdx.y, c0 = blockIdx.x * 64;
  float mx = -INFINITY;
  for (int t = tid; t < L; t += blockDim.x) {
    const float* p = spc + ((int64_t)b * L + t) * np;
    float s = 0.f;
    for (int k = 0; k < np; ++k) s += p[k];
    a[t] = s;
    mx = fmaxf(mx, s);
  }
  mx = wave_max(mx);
  if ((tid & 63) == 0) wr[tid >> 6] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(wr[0], wr[1]), fmaxf(wr[2], wr[3]));
  float sum = 0.f;
  for (int t = tid; t < L; t += blockDim.x) {
    const float e = __expf(a[t] - mx);
    a[t] = e;
    sum += e;
  }
  sum = wave_sum(sum);
  __syncthreads();
  if ((tid & 63) == 0) wr[tid >> 6] = sum;
  __syncthreads();
  const float total = (wr[0] + wr[1]) + (wr[2] + wr[3]);
  const int vi = tid % NV, g = tid / NV;
  float acc[VE];
#pragma unroll
  for (int e = 0; e < VE; ++e) acc[e] = 0.f;
  const T* hb = Hc + (int64_t)b * L * D + c0 + vi * VE;
  constexpr int U = 4;
  for (int t0 = g; t0 < L; t0 += U * G) {
    typename Vec16<T>::type hv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = t0 + u * G;
      hv[u] = t < L ? load16(hb + (int64_t)t * D) : typename Vec16<T>::type{};
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = t0 + u * G;
      const float w = t < L ? a[t] : 0.f;
#pragma unroll
      for (int e = 0; e < VE; ++e) acc[e] += w * to_f32(hv[u][e]);
    }
  }
#pragma unroll
  for (int e = 0; e < VE; ++e) red[g][vi * VE + e] = acc[e];
  __syncthreads();
  if (tid < 64) {
    float S = 0.f;
    for (int k = 0; k < G; ++k) S += red[k][tid];
    S /= total;
    const int64_t o = (int64_t)b * D + c0 + tid;
    const float gam = gvec ? gvec[c0 + tid] : gamma;
    const float nn = gam * N[o] + S;
    N[o] = nn;
    Mt[o] = from_f32<T>(nn / (gam * (gvec ? Z[o] : Z[b]) + 1.f));
  }
}

// K split: enough workgroups to cover the chip (about 256), each taking a
// multiple of 32 rows and at most kDvMaxKc.
int dv_plan(int K, int N, int B, int cols, int* kc) {
  const int tiles = ((N + cols - 1) / cols) * ((B + kDvB - 1) / kDvB);
  const int target = (256 + tiles - 1) / tiles;
  int c = K / target / kDvRowStep * kDvRowStep;
  if (c < kDvRowStep) c = kDvRowStep;
  if (c > kDvMaxKc) c = kDvMaxKc;
  *kc = c;
  return (K + c - 1) / c;
}

}  // namespace

int dec_max_blocklen() { return kDecMaxL; }
int dec_max_batch() { return kDecMaxBatch; }
int dec_score_parts(int D) { return D / 64; }

int dec_splits(DType dt, int K, int N, int B) {
  int kc;
  return dv_plan(K, N, B, dt == DType::BF16 ? dv_cols<bf16>() : dv_cols<float>(), &kc);
}

size_t dec_part_bytes(DType dt, int B, int D) {
  const size_t a = (size_t)dec_splits(dt, D, 3 * D, B) * B * 3 * D;
  const size_t b = (size_t)dec_splits(dt, D, D, B) * B * D;
  return (a > b ? a : b) * sizeof(float);
}

hipError_t dec_product(DType dt, const void* x, int64_t ldx, const void* W0, const void* W1,
                       const void* W2, int B, int D, int N, float* part, hipStream_t s) {
  int kc;
  if (dt == DType::BF16) {
    const int ks = dv_plan(D, N, B, dv_cols<bf16>(), &kc);
    const DvW<bf16> w{{(const bf16*)W0, (const bf16*)(W1 ? W1 : W0), (const bf16*)(W2 ? W2 : W0)},
                      D, D};
    hipLaunchKernelGGL(dec_gemv_part_kernel<bf16>, dim3(N / dv_cols<bf16>(), ks, (B + kDvB - 1) / kDvB),
                       dim3(256), 0, s, (const bf16*)x, ldx, B, w, D, N, kc, part);
  } else {
    const int ks = dv_plan(D, N, B, dv_cols<float>(), &kc);
    const DvW<float> w{
        {(const float*)W0, (const float*)(W1 ? W1 : W0), (const float*)(W2 ? W2 : W0)}, D, D};
    hipLaunchKernelGGL(dec_gemv_part_kernel<float>,
                       dim3(N / dv_cols<float>(), ks, (B + kDvB - 1) / kDvB), dim3(256), 0, s,
                       (const float*)x, ldx, B, w, D, N, kc, part);
  }
  return hipGetLastError();
}

hipError_t dec_attn(DType dt, const float* part, int ks, void* Kc, void* Vc, void* o, int B, int D,
                    int H, int L, int off, hipStream_t s) {
  if (dt == DType::BF16)
    hipLaunchKernelGGL(dec_attn_kernel<bf16>, dim3(H, B), dim3(256), 0, s, part, ks, B,
                       (bf16*)Kc, (bf16*)Vc, (bf16*)o, D, L, off);
  else
    hipLaunchKernelGGL(dec_attn_kernel<float>, dim3(H, B), dim3(256), 0, s, part, ks, B,
                       (float*)Kc, (float*)Vc, (float*)o, D, L, off);
  return hipGetLastError();
}

hipError_t dec_wo_finish(DType dt, const float* part, int ks, const void* wp, void* Hc, float* spc,
                         int B, int D, int L, int off, hipStream_t s) {
  const dim3 grid((D + 255) / 256, B);
  if (dt == DType::BF16)
    hipLaunchKernelGGL(dec_wo_finish_kernel<bf16>, grid, dim3(256), 0, s, part, ks, B, D,
                       (const bf16*)wp, (bf16*)Hc, spc, L, off);
  else
    hipLaunchKernelGGL(dec_wo_finish_kernel<float>, grid, dim3(256), 0, s, part, ks, B, D,
                       (const float*)wp, (float*)Hc, spc, L, off);
  return hipGetLastError();
}

hipError_t dec_gate_finish(DType dt, const float* part, int ks, const void* Hc, const float* C,
                           const void* x, void* y, int B, int D, int L, int off, hipStream_t s) {
  const dim3 grid((D + 255) / 256, B);
  if (dt == DType::BF16)
    hipLaunchKernelGGL(dec_gate_finish_kernel<bf16>, grid, dim3(256), 0, s, part, ks, B, D,
                       (const bf16*)Hc, C, (const bf16*)x, (bf16*)y, L, off);
  else
    hipLaunchKernelGGL(dec_gate_finish_kernel<float>, grid, dim3(256), 0, s, part, ks, B, D,
                       (const float*)Hc, C, (const float*)x, (float*)y, L, off);
  return hipGetLastError();
}

hipError_t dec_mem_finish(const float* part, int ks, float* C, float* Z, int B, int D, float gamma,
                          const float* gvec, hipStream_t s) {
  hipLaunchKernelGGL(dec_mem_finish_kernel, dim3((D + 255) / 256, B), dim3(256), 0, s, part, ks,
                     B, D, C, Z, gamma, gvec);
  return hipGetLastError();
}

hipError_t dec_pool(DType dt, const void* Hc, const float* spc, float* N, const float* Z, void* Mt,
                    int B, int D, int L, float gamma, const float* gvec, hipStream_t s) {
  const int np = dec_score_parts(D);
  if (dt == DType::BF16)
    hipLaunchKernelGGL(dec_pool_kernel<bf16>, dim3(D / 64, B), dim3(256), 0, s, (const bf16*)Hc,
                       spc, np, N, Z, (bf16*)Mt, D, L, gamma, gvec);
  else
    hipLaunchKernelGGL(dec_pool_kernel<float>, dim3(D / 64, B), dim3(256), 0, s, (const float*)Hc,
                       spc, np, N, Z, (float*)Mt, D, L, gamma, gvec);
  return hipGetLastError();
}

}  // namespace bcmt
