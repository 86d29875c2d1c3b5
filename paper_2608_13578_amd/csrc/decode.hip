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
// weight, so they are weight-streaming matrix-vector products: a workgroup
// reads a 32-row by 64-column (bf16) tile of the weight per round, lanes
// owning 16-byte column vectors, and keeps every sequence's partial sums.
// K is split over workgroups; the last workgroup to finish a column tile
// (an atomic ticket per tile, reset by that workgroup) adds the K partials
// in a fixed order and applies the step's epilogue, so each product is one
// launch and its result is the same on every run.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "common.h"
#include "kernels.h"

namespace bcmt {
namespace {

constexpr int kDvB = 8;                     // sequences per workgroup
constexpr int kDvWaves = 4;
constexpr int kDvLanesPerRow = 8;           // a row of the column tile: 8 lanes x 16 bytes
constexpr int kDvRowsPerWave = 64 / kDvLanesPerRow;
constexpr int kDvRowStep = kDvWaves * kDvRowsPerWave;  // rows per round (32)
constexpr int kDvMaxKc = 256;               // K rows per workgroup at most
constexpr int kDvUnroll = 4;                // rounds whose loads are issued together
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

template <typename T, class Epi>
__global__ __launch_bounds__(kDvWaves * 64) void dec_gemv_kernel(
    const T* __restrict__ x, int64_t ldx, int B, DvW<T> w, int K, int N, int kc,
    float* __restrict__ part, unsigned* __restrict__ tickets, Epi epi) {
  constexpr int VE = Vec16<T>::N, CT = dv_cols<T>();
  __shared__ float xs[kDvB][kDvMaxKc];
  __shared__ float red[kDvWaves][kDvB][CT];
  __shared__ float vals[kDvB][CT];
  __shared__ int last;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n0 = blockIdx.x * CT;
  const int k0 = blockIdx.y * kc;
  const int b0 = blockIdx.z * kDvB;
  const int nbt = min(kDvB, B - b0);
  const int kn = min(kc, K - k0);
  // Every entry is written (zeros past the rows and sequences present), so
  // the rounds past kn multiply zero weights by zeros.
  for (int e = tid; e < kDvB * kDvMaxKc; e += blockDim.x) {
    const int b = e / kDvMaxKc, k = e % kDvMaxKc;
    xs[b][k] = (b < nbt && k < kn) ? to_f32(x[(int64_t)(b0 + b) * ldx + k0 + k]) : 0.f;
  }
  __syncthreads();
  const int cg = lane % kDvLanesPerRow, rl = lane / kDvLanesPerRow;
  const T* wcol = w.col(n0 + cg * VE);
  float acc[kDvB][VE];
#pragma unroll
  for (int b = 0; b < kDvB; ++b)
#pragma unroll
    for (int e = 0; e < VE; ++e) acc[b][e] = 0.f;
  for (int r0 = wave * kDvRowsPerWave + rl; r0 < kn; r0 += kDvUnroll * kDvRowStep) {
    typename Vec16<T>::type wv[kDvUnroll];
#pragma unroll
    for (int u = 0; u < kDvUnroll; ++u) {
      const int r = r0 + u * kDvRowStep;
      wv[u] = r < kn ? load16(wcol + (int64_t)(k0 + r) * w.ld) : typename Vec16<T>::type{};
    }
#pragma unroll
    for (int u = 0; u < kDvUnroll; ++u) {
      const int r = min(r0 + u * kDvRowStep, kDvMaxKc - 1);  // zero weights past kn
#pragma unroll
      for (int b = 0; b < kDvB; ++b) {
        const float xb = xs[b][r];
#pragma unroll
        for (int e = 0; e < VE; ++e) acc[b][e] += xb * to_f32(wv[u][e]);
      }
    }
  }
  // Lanes of one column vector (same cg) hold different rows: add them up.
#pragma unroll
  for (int b = 0; b < kDvB; ++b)
#pragma unroll
    for (int e = 0; e < VE; ++e) {
      float v = acc[b][e];
      v += __shfl_xor(v, 8);
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (rl == 0) red[wave][b][cg * VE + e] = v;
    }
  __syncthreads();
  for (int e = tid; e < kDvB * CT; e += blockDim.x) {
    const int b = e / CT, c = e % CT;
    const float v = (red[0][b][c] + red[1][b][c]) + (red[2][b][c] + red[3][b][c]);
    if (b < nbt && n0 + c < N) part[((int64_t)blockIdx.y * B + b0 + b) * N + n0 + c] = v;
  }
  // Publish the partials, then take a ticket; the last of the K splits of
  // this tile finishes it.
  __threadfence();
  __syncthreads();
  unsigned* tk = tickets + blockIdx.z * gridDim.x + blockIdx.x;
  if (tid == 0) last = atomicAdd(tk, 1u) == gridDim.y - 1;
  __syncthreads();
  if (!last) return;
  __threadfence();
  for (int e = tid; e < kDvB * CT; e += blockDim.x) {
    const int b = e / CT, c = e % CT;
    float v = 0.f;
    if (b < nbt && n0 + c < N)
      for (int s = 0; s < (int)gridDim.y; ++s) v += part[((int64_t)s * B + b0 + b) * N + n0 + c];
    vals[b][c] = v;
  }
  if (tid == 0) *tk = 0u;  // ready for the next product
  __syncthreads();
  epi.finish(b0, nbt, n0, vals, tid);
}

// [q k v]: q to its buffer, k and v to the block caches at slot `off`.
template <typename T>
struct EpiDecQkv {
  T* q;
  T* Kc;
  T* Vc;
  int D, L, off;
  template <int CT>
  __device__ void finish(int b0, int nbt, int n0, const float (&v)[kDvB][CT], int tid) const {
    for (int e = tid; e < nbt * CT; e += blockDim.x) {
      const int b = e / CT, c = e % CT, n = n0 + c;
      const int sg = n / D, col = n - sg * D;
      const T val = from_f32<T>(v[b][c]);
      if (sg == 0) q[(int64_t)(b0 + b) * D + col] = val;
      else (sg == 1 ? Kc : Vc)[((int64_t)(b0 + b) * L + off) * D + col] = val;
    }
  }
};

// h = o Wo to the block cache, and this tile's part of the score h . wp.
template <typename T>
struct EpiDecWo {
  T* Hc;
  float* spc;  // [B, L, np]
  const T* wp;
  int D, L, off, np;
  template <int CT>
  __device__ void finish(int b0, int nbt, int n0, const float (&v)[kDvB][CT], int tid) const {
    for (int e = tid; e < nbt * CT; e += blockDim.x) {
      const int b = e / CT, c = e % CT;
      Hc[((int64_t)(b0 + b) * L + off) * D + n0 + c] = from_f32<T>(v[b][c]);
    }
    if (tid < nbt) {
      float sc = 0.f;
      for (int c = 0; c < CT; ++c) sc += v[tid][c] * to_f32(wp[n0 + c]);
      spc[((int64_t)(b0 + tid) * L + off) * np + n0 / CT] = sc;
    }
  }
};

// y = h + sigmoid(u) * C (+ x), u = h Wg.
template <typename T>
struct EpiDecGate {
  T* y;
  const T* Hc;
  const float* C;
  const T* x;  // nullable
  int D, L, off;
  template <int CT>
  __device__ void finish(int b0, int nbt, int n0, const float (&v)[kDvB][CT], int tid) const {
    for (int e = tid; e < nbt * CT; e += blockDim.x) {
      const int b = e / CT, c = e % CT, n = n0 + c;
      const int64_t row = (int64_t)(b0 + b) * D + n;
      float out = to_f32(Hc[((int64_t)(b0 + b) * L + off) * D + n]) + sigmoidf_(v[b][c]) * C[row];
      if (x) out += to_f32(x[row]);
      y[row] = from_f32<T>(out);
    }
  }
};

// C = Mt Wm for the next block; the first column tile also advances Z.
struct EpiDecMem {
  float* C;
  float* Z;
  int D;
  float gamma;
  template <int CT>
  __device__ void finish(int b0, int nbt, int n0, const float (&v)[kDvB][CT], int tid) const {
    for (int e = tid; e < nbt * CT; e += blockDim.x) {
      const int b = e / CT, c = e % CT;
      C[(int64_t)(b0 + b) * D + n0 + c] = v[b][c];
    }
    if (n0 == 0 && tid < nbt) Z[b0 + tid] = gamma * Z[b0 + tid] + 1.f;
  }
};

// Attention of the new token over the block's cached tokens 0..off, one
// workgroup per (head, sequence): scores one key per thread, then thread
// (dim d, key group g) adds p_j V[j, d] over the keys j = g mod 4.
constexpr int kDecMaxL = 4096;

template <typename T>
__global__ __launch_bounds__(256) void dec_attn_kernel(const T* __restrict__ q,
                                                       const T* __restrict__ Kc,
                                                       const T* __restrict__ Vc,
                                                       T* __restrict__ o, int D, int L, int off) {
  constexpr int VE = Vec16<T>::N;
  __shared__ float qs[64];
  __shared__ float sc[kDecMaxL];
  __shared__ float red[4][64];
  __shared__ float wr[4];
  const int tid = threadIdx.x, h = blockIdx.x, b = blockIdx.y;
  const int n = off + 1;
  if (tid < 64) qs[tid] = to_f32(q[(int64_t)b * D + h * 64 + tid]) * 0.125f;
  __syncthreads();
  float mx = -INFINITY;
  for (int j = tid; j < n; j += blockDim.x) {
    const T* kr = Kc + ((int64_t)b * L + j) * D + h * 64;
    float d = 0.f;
#pragma unroll
    for (int v = 0; v < 64 / VE; ++v) {
      const auto kv = load16(kr + v * VE);
#pragma unroll
      for (int e = 0; e < VE; ++e) d += qs[v * VE + e] * to_f32(kv[e]);
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
  const int d = tid & 63, g = tid >> 6;
  float acc = 0.f;
  for (int j = g; j < n; j += 4) acc += sc[j] * to_f32(Vc[((int64_t)b * L + j) * D + h * 64 + d]);
  red[g][d] = acc;
  __syncthreads();
  if (tid < 64)
    o[(int64_t)b * D + h * 64 + tid] =
        from_f32<T>(((red[0][tid] + red[1][tid]) + (red[2][tid] + red[3][tid])) / total);
}

// After a block's last token: a = softmax of the block's scores, S = sum_t
// a_t H[t] for 64 columns per workgroup, N = g N + S, and the new memory
// N / (g Z + 1) in the compute type (Z itself advances in the W_m product).
template <typename T>
__global__ __launch_bounds__(256) void dec_pool_kernel(const T* __restrict__ Hc,
                                                       const float* __restrict__ spc, int np,
                                                       float* __restrict__ N,
                                                       const float* __restrict__ Z,
                                                       T* __restrict__ Mt, int D, int L,
                                                       float gamma) {
  __shared__ float a[kDecMaxL];
  __shared__ float red[4][64];
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
  const int d = tid & 63, g = tid >> 6;
  float acc = 0.f;
  for (int t = g; t < L; t += 4) acc += a[t] * to_f32(Hc[((int64_t)b * L + t) * D + c0 + d]);
  red[g][d] = acc;
  __syncthreads();
  if (tid < 64) {
    const int64_t o = (int64_t)b * D + c0 + tid;
    const float S = ((red[0][tid] + red[1][tid]) + (red[2][tid] + red[3][tid])) / total;
    const float nn = gamma * N[o] + S;
    N[o] = nn;
    Mt[o] = from_f32<T>(nn / (gamma * Z[b] + 1.f));
  }
}

// Split of K over workgroups: enough workgroups to cover the chip, each
// taking a multiple of 32 rows and at most kDvMaxKc.
int dv_plan(int K, int N, int B, int cols, int* kc) {
  const int tiles = ((N + cols - 1) / cols) * ((B + kDvB - 1) / kDvB);
  int ks = (256 + tiles - 1) / tiles;
  if (ks > K / kDvRowStep) ks = K / kDvRowStep;
  if (ks < 1) ks = 1;
  int c = (K + ks - 1) / ks;
  c = (c + kDvRowStep - 1) / kDvRowStep * kDvRowStep;
  if (c > kDvMaxKc) c = kDvMaxKc;
  *kc = c;
  return (K + c - 1) / c;
}

template <typename T, class Epi>
hipError_t dv_launch(const T* x, int64_t ldx, int B, DvW<T> w, int K, int N, float* part,
                     unsigned* tickets, const Epi& epi, hipStream_t s) {
  constexpr int CT = dv_cols<T>();
  int kc;
  const int ks = dv_plan(K, N, B, CT, &kc);
  dim3 grid((N + CT - 1) / CT, ks, (B + kDvB - 1) / kDvB);
  hipLaunchKernelGGL((dec_gemv_kernel<T, Epi>), grid, dim3(kDvWaves * 64), 0, s, x, ldx, B, w, K,
                     N, kc, part, tickets, epi);
  return hipGetLastError();
}

template <typename T>
DvW<T> dv_w(const void* a, const void* b, const void* c, int seg, int64_t ld) {
  return DvW<T>{{(const T*)a, (const T*)(b ? b : a), (const T*)(c ? c : a)}, seg, ld};
}

}  // namespace

int dec_max_blocklen() { return kDecMaxL; }
int dec_max_batch() { return kDecMaxBatch; }

int dec_score_parts(DType dt, int D) {
  return D / (dt == DType::BF16 ? dv_cols<bf16>() : dv_cols<float>());
}

size_t dec_part_bytes(DType dt, int B, int D) {
  const int cols = dt == DType::BF16 ? dv_cols<bf16>() : dv_cols<float>();
  int kc;
  const size_t a = (size_t)dv_plan(D, 3 * D, B, cols, &kc) * B * 3 * D;
  const size_t b = (size_t)dv_plan(D, D, B, cols, &kc) * B * D;
  return (a > b ? a : b) * sizeof(float);
}

hipError_t dec_qkv(DType dt, const void* x, const void* Wq, const void* Wk, const void* Wv,
                   void* q, void* Kc, void* Vc, int B, int D, int L, int off, float* part,
                   unsigned* tickets, hipStream_t s) {
  if (dt == DType::BF16)
    return dv_launch<bf16>((const bf16*)x, D, B, dv_w<bf16>(Wq, Wk, Wv, D, D), D, 3 * D, part,
                           tickets, EpiDecQkv<bf16>{(bf16*)q, (bf16*)Kc, (bf16*)Vc, D, L, off}, s);
  return dv_launch<float>((const float*)x, D, B, dv_w<float>(Wq, Wk, Wv, D, D), D, 3 * D, part,
                          tickets, EpiDecQkv<float>{(float*)q, (float*)Kc, (float*)Vc, D, L, off},
                          s);
}

hipError_t dec_attn(DType dt, const void* q, const void* Kc, const void* Vc, void* o, int B,
                    int D, int H, int L, int off, hipStream_t s) {
  if (dt == DType::BF16)
    hipLaunchKernelGGL(dec_attn_kernel<bf16>, dim3(H, B), dim3(256), 0, s, (const bf16*)q,
                       (const bf16*)Kc, (const bf16*)Vc, (bf16*)o, D, L, off);
  else
    hipLaunchKernelGGL(dec_attn_kernel<float>, dim3(H, B), dim3(256), 0, s, (const float*)q,
                       (const float*)Kc, (const float*)Vc, (float*)o, D, L, off);
  return hipGetLastError();
}

hipError_t dec_wo(DType dt, const void* o, const void* Wo, const void* wp, void* Hc, float* spc,
                  int B, int D, int L, int off, float* part, unsigned* tickets, hipStream_t s) {
  const int np = dec_score_parts(dt, D);
  if (dt == DType::BF16)
    return dv_launch<bf16>((const bf16*)o, D, B, dv_w<bf16>(Wo, nullptr, nullptr, D, D), D, D,
                           part, tickets,
                           EpiDecWo<bf16>{(bf16*)Hc, spc, (const bf16*)wp, D, L, off, np}, s);
  return dv_launch<float>((const float*)o, D, B, dv_w<float>(Wo, nullptr, nullptr, D, D), D, D,
                          part, tickets,
                          EpiDecWo<float>{(float*)Hc, spc, (const float*)wp, D, L, off, np}, s);
}

hipError_t dec_gate(DType dt, const void* Wg, const void* Hc, const float* C, const void* x,
                    void* y, int B, int D, int L, int off, float* part, unsigned* tickets,
                    hipStream_t s) {
  const int64_t ldh = (int64_t)L * D;
  if (dt == DType::BF16) {
    const bf16* h = (const bf16*)Hc + (int64_t)off * D;
    return dv_launch<bf16>(h, ldh, B, dv_w<bf16>(Wg, nullptr, nullptr, D, D), D, D, part, tickets,
                           EpiDecGate<bf16>{(bf16*)y, (const bf16*)Hc, C, (const bf16*)x, D, L,
                                            off}, s);
  }
  const float* h = (const float*)Hc + (int64_t)off * D;
  return dv_launch<float>(h, ldh, B, dv_w<float>(Wg, nullptr, nullptr, D, D), D, D, part, tickets,
                          EpiDecGate<float>{(float*)y, (const float*)Hc, C, (const float*)x, D, L,
                                            off}, s);
}

hipError_t dec_pool(DType dt, const void* Hc, const float* spc, float* N, const float* Z, void* Mt,
                    int B, int D, int L, float gamma, hipStream_t s) {
  const int np = dec_score_parts(dt, D);
  if (dt == DType::BF16)
    hipLaunchKernelGGL(dec_pool_kernel<bf16>, dim3(D / 64, B), dim3(256), 0, s, (const bf16*)Hc,
                       spc, np, N, Z, (bf16*)Mt, D, L, gamma);
  else
    hipLaunchKernelGGL(dec_pool_kernel<float>, dim3(D / 64, B), dim3(256), 0, s, (const float*)Hc,
                       spc, np, N, Z, (float*)Mt, D, L, gamma);
  return hipGetLastError();
}

hipError_t dec_mem(DType dt, const void* Mt, const void* Wm, float* C, float* Z, int B, int D,
                   float gamma, float* part, unsigned* tickets, hipStream_t s) {
  if (dt == DType::BF16)
    return dv_launch<bf16>((const bf16*)Mt, D, B, dv_w<bf16>(Wm, nullptr, nullptr, D, D), D, D,
                           part, tickets, EpiDecMem{C, Z, D, gamma}, s);
  return dv_launch<float>((const float*)Mt, D, B, dv_w<float>(Wm, nullptr, nullptr, D, D), D, D,
                          part, tickets, EpiDecMem{C, Z, D, gamma}, s);
}

}  // namespace bcmt
