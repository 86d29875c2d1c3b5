// Tiled matrix products on the CDNA4 matrix cores, with fused epilogues.
//
// Serves every dense projection of the layer (Sec. 3.3 Q/K/V and W_O,
// Sec. 3.5 W_m, Sec. 3.8 W_g) and their backward products.
//
// Two kernels:
//  * gemm_pipe_kernel (bf16): 128 x 128 tiles, four waves of 64 x 64, K
//    streamed in 64-deep slabs through a two-slab LDS ring filled by direct
//    global->LDS loads; operands stay in their global orientation in LDS and
//    M/N-major ones are read with the transposing LDS instruction.  Two
//    workgroups share a CU.  Tiles are ordered per XCD (see xcd_tile_order).
//  * gemm_kernel (float32, and bf16 shapes whose K is not a multiple of 64):
//    the same tiling with register staging; M/N-major operands are
//    transposed in registers on their way into LDS.
// Weight gradients (K = B*T) use split-K partial tiles and a deterministic
// reduction kernel instead of atomics.
//
// The matrix instruction is issued with the B tile as its first operand, so
// a lane ends up holding four consecutive output columns of one output row:
// the epilogue stores 8 (bf16) or 16 (f32) contiguous bytes per lane.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace bcmt {
namespace {

constexpr int kThreads = 256;
constexpr int BM = 128;
constexpr int BN = 128;

template <typename T> struct KSlab;
template <> struct KSlab<bf16> { static constexpr int BK = 64; };
template <> struct KSlab<float> { static constexpr int BK = 32; };

// An operand indexed by (row, k), where row is m for A and n for B.
template <typename T, bool RCONTIG, int SEG>
struct Operand {
  const T* p[3];
  int64_t ld;
  int seg_len;
  __device__ __forceinline__ const T* at(int row, int k) const {
    int s = 0;
    if constexpr (SEG == kSegN) {
      s = row / seg_len;
      row -= s * seg_len;
    } else if constexpr (SEG == kSegK) {
      s = k / seg_len;
      k -= s * seg_len;
    }
    return p[s] + (RCONTIG ? (int64_t)k * ld + row : (int64_t)row * ld + k);
  }
};

// Registers holding one operand's share of a K slab between its global load
// and its LDS store.
template <typename T, bool RCONTIG, int SEG, int R>
struct Stage {
  static constexpr int VE = Vec16<T>::N;
  static constexpr int BK = KSlab<T>::BK;
  static constexpr int LDS_ROW = BK + VE;
  typedef typename Vec16<T>::type vec;
  // K-contiguous: R rows of BK/VE vectors.  Row-contiguous: (BK/VE) x (R/VE)
  // sub-blocks of VE x VE elements, at most one per thread.
  static constexpr int NV = RCONTIG ? VE : (R * (BK / VE)) / kThreads;
  static constexpr int NSB = (BK / VE) * (R / VE);
  static_assert(RCONTIG ? NSB <= kThreads : (R * (BK / VE)) % kThreads == 0, "tile");
  vec r[NV];

  __device__ __forceinline__ void load(const Operand<T, RCONTIG, SEG>& op, int row0, int rmax,
                                       int k0, int kend, int tid) {
    if constexpr (!RCONTIG) {
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int idx = tid + v * kThreads;
        const int rr = idx / (BK / VE);
        const int cc = (idx % (BK / VE)) * VE;
        const int gr = row0 + rr, gk = k0 + cc;
        if (gr < rmax && gk < kend) r[v] = load16(op.at(gr, gk));
        else r[v] = vec{};
      }
    } else {
      if (tid < NSB) {
        const int kb = tid / (R / VE);
        const int rb = tid % (R / VE);
        const int gr = row0 + rb * VE;
#pragma unroll
        for (int j = 0; j < VE; ++j) {
          const int gk = k0 + kb * VE + j;
          if (gr < rmax && gk < kend) r[j] = load16(op.at(gr, gk));
          else r[j] = vec{};
        }
      }
    }
  }

  __device__ __forceinline__ void store(T* lds, int tid) const {
    if constexpr (!RCONTIG) {
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int idx = tid + v * kThreads;
        const int rr = idx / (BK / VE);
        const int cc = (idx % (BK / VE)) * VE;
        store16(lds + rr * LDS_ROW + cc, r[v]);
      }
    } else {
      if (tid < NSB) {
        const int kb = tid / (R / VE);
        const int rb = tid % (R / VE);
#pragma unroll
        for (int i = 0; i < VE; ++i) {
          vec t;
#pragma unroll
          for (int j = 0; j < VE; ++j) t[j] = r[j][i];
          store16(lds + (rb * VE + i) * LDS_ROW + kb * VE, t);
        }
      }
    }
  }
};

template <typename T, bool A_MC, bool B_NC, int BSEG, class Epi>
__global__ __launch_bounds__(kThreads) void gemm_kernel(int M, int N, int K,
                                                        Operand<T, A_MC, kSegNone> A,
                                                        Operand<T, B_NC, BSEG> B, int kchunk,
                                                        Epi epi0) {
  constexpr int BK = KSlab<T>::BK;
  constexpr int VE = Vec16<T>::N;
  constexpr int LDS_ROW = BK + VE;
  __shared__ __attribute__((aligned(16))) T As[2][BM * LDS_ROW];
  __shared__ __attribute__((aligned(16))) T Bs[2][BN * LDS_ROW];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int lr = lane & 15, lg = lane >> 4;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int kbeg = blockIdx.z * kchunk;
  Epi epi = epi0;
  bind_split(epi, blockIdx.z);
  const int kend = min(K, kbeg + kchunk);
  const int nk = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;

  Stage<T, A_MC, kSegNone, BM> sa;
  Stage<T, B_NC, BSEG, BN> sb;
  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (nk > 0) {
    sa.load(A, m0, M, kbeg, kend, tid);
    sb.load(B, n0, N, kbeg, kend, tid);
    sa.store(As[0], tid);
    sb.store(Bs[0], tid);
  }
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
      const int k0 = kbeg + (kt + 1) * BK;
      sa.load(A, m0, M, k0, kend, tid);
      sb.load(B, n0, N, k0, kend, tid);
    }
    const T* as = As[cur];
    const T* bs = Bs[cur];
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      typename Frag<T>::type fa[4], fb[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        fa[i] = load_frag(as + (wm * 64 + i * 16 + lr) * LDS_ROW + ks * 32 + lg * 8);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        fb[j] = load_frag(bs + (wn * 64 + j * 16 + lr) * LDS_ROW + ks * 32 + lg * 8);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mma16(fb[j], fa[i], acc[i][j]);
    }
    if (more) {
      sa.store(As[cur ^ 1], tid);
      sb.store(Bs[cur ^ 1], tid);
    }
    __syncthreads();
  }

  run_epilogue<4, 4>(epi, acc, m0 + wm * 64, n0 + wn * 64, M, N, lane);
}

// ------------------------------------------------------------------ epilogue driver
// Hands every fragment of a wave's tile to the epilogue.  An epilogue with
// kRowDot also folds each fragment into a per-row value (rowdot) that is
// summed over the wave's columns and handed to row() once per row, by the
// lane group holding the row's first four columns.
template <class Epi, class = void>
struct HasRowDot {
  static constexpr bool value = false;
};
template <class Epi>
struct HasRowDot<Epi, decltype((void)Epi::kRowDot)> {
  static constexpr bool value = Epi::kRowDot;
};

template <int FM, int FN, class Epi>
__device__ __forceinline__ void run_epilogue(const Epi& epi, const f32x4 (&acc)[FM][FN], int mb,
                                             int nb, int M, int N, int lane) {
  const int lr = lane & 15, lg = lane >> 4;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int m = mb + i * 16 + lr;
    float rs = 0.f;
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int n = nb + j * 16 + lg * 4;
      if (m < M && n < N) {
        epi(m, n, acc[i][j]);
        if constexpr (HasRowDot<Epi>::value) rs += epi.rowdot(n, acc[i][j]);
      }
    }
    if constexpr (HasRowDot<Epi>::value) {
      rs += __shfl_xor(rs, 16);
      rs += __shfl_xor(rs, 32);
      if (lg == 0 && m < M && nb < N) epi.row(m, nb, rs);
    }
  }
}

// 8 consecutive elements to / from float (16 bytes of bf16, 32 of float).
// Staged epilogue of the pipelined kernel.  The accumulator tile goes to
// LDS (float32, rows of BN, 16-byte chunks XOR-swizzled by row so that the
// 16 rows a fragment spans fall on distinct banks), then every thread hands
// 8 consecutive columns of a row at a time to the epilogue's apply8: the
// 16 lanes of a row write one contiguous 256-byte (bf16) segment, where the
// fragment layout would write 32-byte pieces of 16 rows.  Every lane calls
// apply8 the same number of times (with ok = false outside the matrix), so
// an epilogue may reduce across lanes.
template <int BM, int BN, int FM, int FN, int WTM, int WTN, int NTH, class Epi>
__device__ __forceinline__ void staged_epilogue(const Epi& epi, const f32x4 (&acc)[FM][FN],
                                                float* cs, int m0, int n0, int wm, int wn, int M,
                                                int N, int tid) {
  constexpr int CH = BN / 4;  // 16-byte chunks per row
  static_assert((CH & (CH - 1)) == 0, "power-of-two row chunks");
  const int lane = tid & 63, lr = lane & 15, lg = lane >> 4;
  __syncthreads();  // every wave is done reading the operand slabs
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int r = wm * WTM + i * 16 + lr;
      const int c4 = (wn * WTN + j * 16 + lg * 4) / 4;
      *reinterpret_cast<f32x4*>(cs + r * BN + ((c4 ^ (r & (CH - 1))) * 4)) = acc[i][j];
    }
  __syncthreads();
  constexpr int CPR = BN / 8;  // 8-column items per row
  static_assert((BM * CPR) % NTH == 0, "items per thread");
#pragma unroll 2
  for (int it = tid; it < BM * CPR; it += NTH) {
    const int r = it / CPR, c8 = it % CPR;
    const float* row = cs + r * BN;
    const f32x4 a = *reinterpret_cast<const f32x4*>(row + (((2 * c8) ^ (r & (CH - 1))) * 4));
    const f32x4 b = *reinterpret_cast<const f32x4*>(row + (((2 * c8 + 1) ^ (r & (CH - 1))) * 4));
    const float v[8] = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    const int m = m0 + r, n = n0 + c8 * 8;
    epi.apply8(m, n, v, m < M && n < N);
  }
}

// ------------------------------------------------------------------ epilogues

template <typename TO, typename TA>
struct EpiStore {
  TO* C;
  int64_t ldc;
  const TA* add;
  int64_t ld_add;
  __device__ __forceinline__ void operator()(int m, int n, f32x4 v) const {
    if (add) v += load4f(add + (int64_t)m * ld_add + n);
    store4(C + (int64_t)m * ldc + n, v[0], v[1], v[2], v[3]);
  }
  __device__ __forceinline__ void apply8(int m, int n, const float (&v)[8], bool ok) const {
    if (!ok) return;
    float o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = v[e];
    if (add) {
      float a[8];
      ld8(add + (int64_t)m * ld_add + n, a);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] += a[e];
    }
    st8(C + (int64_t)m * ldc + n, o);
  }
};

// GELU, tanh form, and its derivative (the MLP of the language model).
__device__ __forceinline__ float gelu_f(float u) {
  const float c = 0.7978845608028654f;  // sqrt(2 / pi)
  return 0.5f * u * (1.f + tanhf(c * (u + 0.044715f * u * u * u)));
}
__device__ __forceinline__ float gelu_grad_f(float u) {
  const float c = 0.7978845608028654f;
  const float t = tanhf(c * (u + 0.044715f * u * u * u));
  return 0.5f * (1.f + t) + 0.5f * u * (1.f - t * t) * c * (1.f + 3.f * 0.044715f * u * u);
}

// MLP input product: stores U = acc (rounded to T, kept for the backward)
// and A = gelu(U) of the rounded U.
template <typename T>
struct EpiGelu {
  T* U;
  T* A;
  int64_t ld;
  __device__ __forceinline__ void operator()(int m, int n, f32x4 v) const {
    const int64_t off = (int64_t)m * ld + n;
    f32x4 a;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      v[r] = (float)(T)v[r];
      a[r] = gelu_f(v[r]);
    }
    store4(U + off, v[0], v[1], v[2], v[3]);
    store4(A + off, a[0], a[1], a[2], a[3]);
  }
  __device__ __forceinline__ void apply8(int m, int n, const float (&v)[8], bool ok) const {
    if (!ok) return;
    const int64_t off = (int64_t)m * ld + n;
    float u[8], a[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      u[k] = (float)(T)v[k];
      a[k] = gelu_f(u[k]);
    }
    st8(U + off, u);
    st8(A + off, a);
  }
};

// Backward through the GELU: dU = acc * gelu'(U), U the stored forward value.
template <typename T>
struct EpiGeluBwd {
  const T* U;
  T* dU;
  int64_t ld;
  __device__ __forceinline__ void operator()(int m, int n, f32x4 v) const {
    const int64_t off = (int64_t)m * ld + n;
    const f32x4 u = load4f(U + off);
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] *= gelu_grad_f(u[r]);
    store4(dU + off, v[0], v[1], v[2], v[3]);
  }
  __device__ __forceinline__ void apply8(int m, int n, const float (&v)[8], bool ok) const {
    if (!ok) return;
    const int64_t off = (int64_t)m * ld + n;
    float u[8], d[8];
    ld8(U + off, u);
#pragma unroll
    for (int k = 0; k < 8; ++k) d[k] = v[k] * gelu_grad_f(u[k]);
    st8(dU + off, d);
  }
};

// Output projection (Sec. 3.3) with the pooling scores of Sec. 3.4 folded
// in: stores H and, for every row, the partial score over this wave's 64
// columns, sum_n H[m, n] wp[n] (from the stored, rounded H), to
// sp[m * (N / 64) + n0 / 64]; the pooling kernel adds the N / 64 parts.
template <typename T>
struct EpiScore {
  T* C;
  int64_t ldc;
  const T* wp;
  float* sp;
  int nparts;
  static constexpr bool kRowDot = true;
  __device__ __forceinline__ void operator()(int m, int n, f32x4 v) const {
    store4(C + (int64_t)m * ldc + n, v[0], v[1], v[2], v[3]);
  }
  __device__ __forceinline__ float rowdot(int n, f32x4 v) const {
    const f32x4 w = load4f(wp + n);
    float d = 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) d += to_f32(from_f32<T>(v[r])) * w[r];
    return d;
  }
  __device__ __forceinline__ void row(int m, int n0, float v) const {
    sp[(int64_t)m * nparts + n0 / 64] = v;
  }
  // The 8 lanes holding one row's 64-column group (n0 a multiple of 64) are
  // consecutive and aligned, so the group's dot is a reduction over them.
  __device__ __forceinline__ void apply8(int m, int n, const float (&v)[8], bool ok) const {
    float d = 0.f;
    if (ok) {
      float o[8], w[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = to_f32(from_f32<T>(v[e]));
      ld8(wp + n, w);
#pragma unroll
      for (int e = 0; e < 8; ++e) d += o[e] * w[e];
      st8(C + (int64_t)m * ldc + n, o);
    }
    d += __shfl_xor(d, 1);
    d += __shfl_xor(d, 2);
    d += __shfl_xor(d, 4);
    if (ok && (n & 63) == 0) sp[(int64_t)m * nparts + n / 64] = d;
  }
};

// Split-K partial tile: split z of an M x N product goes to P + z * M * N
// (the kernel moves P to its split's slice through bind_split).
struct EpiPartial {
  float* P;
  int64_t ld;
  int64_t split_stride;
  __device__ __forceinline__ void operator()(int m, int n, f32x4 v) const {
    store4(P + (int64_t)m * ld + n, v[0], v[1], v[2], v[3]);
  }
  __device__ __forceinline__ void apply8(int m, int n, const float (&v)[8], bool ok) const {
    if (ok) st8(P + (int64_t)m * ld + n, v);
  }
};
__device__ __forceinline__ void bind_split(EpiPartial& e, int z) { e.P += z * e.split_stride; }

// Sums the split-K partials and writes or accumulates into the output
// segment that holds each column.  Workgroup = 64 consecutive groups of 4
// columns; its four waves take the splits z = w, w + 4, ... of their group
// (each in increasing z), and the four sums are added in a fixed order.
__global__ __launch_bounds__(256) void wgrad_reduce_kernel(const float* __restrict__ P, int splits,
                                                           int M, int N, float* C0, float* C1,
                                                           float* C2, int64_t ldc, int seg,
                                                           int accumulate) {
  __shared__ f32x4 red[4][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t total = (int64_t)M * N / 4;
  const int64_t stride = (int64_t)M * N;
  const int64_t i = (int64_t)blockIdx.x * 64 + lane;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  if (i < total) {
    // four of this wave's splits in flight at a time, added in increasing z
    const float* p = P + i * 4;
    int z = wave;
    for (; z + 12 < splits; z += 16) {
      const f32x4 a0 = *reinterpret_cast<const f32x4*>(p + z * stride);
      const f32x4 a1 = *reinterpret_cast<const f32x4*>(p + (z + 4) * stride);
      const f32x4 a2 = *reinterpret_cast<const f32x4*>(p + (z + 8) * stride);
      const f32x4 a3 = *reinterpret_cast<const f32x4*>(p + (z + 12) * stride);
      acc += a0;
      acc += a1;
      acc += a2;
      acc += a3;
    }
    for (; z < splits; z += 4) acc += *reinterpret_cast<const f32x4*>(p + z * stride);
  }
  red[wave][lane] = acc;
  __syncthreads();
  if (wave != 0 || i >= total) return;
  acc = (red[0][lane] + red[1][lane]) + (red[2][lane] + red[3][lane]);
  const int64_t e = i * 4;
  const int m = (int)(e / N), n = (int)(e - (int64_t)m * N);
  const int sg = n / seg;
  float* base = sg == 0 ? C0 : sg == 1 ? C1 : C2;
  if (!base) return;
  f32x4* dst = reinterpret_cast<f32x4*>(base + (int64_t)m * ldc + (n - sg * seg));
  if (accumulate) acc += *dst;
  *dst = acc;
}

template <typename T>
struct EpiGate {
  GateEpi e;
  __device__ __forceinline__ void operator()(int m, int n, f32x4 u) const {
    const int b = m / e.T;
    const int t = m - b * e.T;
    const int blk = t / e.L;
    const int64_t off = (int64_t)m * e.D + n;
    const f32x4 h = load4f(reinterpret_cast<const T*>(e.H) + off);
    f32x4 c = {0.f, 0.f, 0.f, 0.f};
    if (blk > 0) c = load4f(e.P + (int64_t)(b * e.nb + blk - 1) * e.D + n);
    else if (e.Pc) c = load4f(e.Pc + (int64_t)b * e.D + n);
    f32x4 x = {0.f, 0.f, 0.f, 0.f};
    if (e.X) x = load4f(reinterpret_cast<const T*>(e.X) + off);
    f32x4 g, y;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      g[r] = sigmoidf_(u[r]);
      y[r] = h[r] + g[r] * c[r] + x[r];
    }
    store4(reinterpret_cast<T*>(e.Y) + off, y[0], y[1], y[2], y[3]);
    store4(reinterpret_cast<typename GateT<T>::type*>(e.G) + off, g[0], g[1], g[2], g[3]);
  }
  __device__ __forceinline__ void apply8(int m, int n, const float (&u)[8], bool ok) const {
    if (!ok) return;
    const int b = m / e.T;
    const int t = m - b * e.T;
    const int blk = t / e.L;
    const int64_t off = (int64_t)m * e.D + n;
    float h[8], c[8], g[8], y[8];
    ld8(reinterpret_cast<const T*>(e.H) + off, h);
    if (blk > 0) {
      ld8(e.P + (int64_t)(b * e.nb + blk - 1) * e.D + n, c);
    } else if (e.Pc) {
      ld8(e.Pc + (int64_t)b * e.D + n, c);
    } else {
#pragma unroll
      for (int k = 0; k < 8; ++k) c[k] = 0.f;
    }
    if (e.X) {
      float x[8];
      ld8(reinterpret_cast<const T*>(e.X) + off, x);
#pragma unroll
      for (int k = 0; k < 8; ++k) h[k] += x[k];
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      g[k] = sigmoidf_(u[k]);
      y[k] = h[k] + g[k] * c[k];
    }
    st8(reinterpret_cast<T*>(e.Y) + off, y);
    st8(reinterpret_cast<typename GateT<T>::type*>(e.G) + off, g);
  }
};

template <typename T>
struct EpiHbar {
  HbarEpi e;
  __device__ __forceinline__ void operator()(int m, int n, f32x4 v) const {
    const int b = m / e.T;
    const int t = m - b * e.T;
    const int blk = t / e.L;
    const int64_t off = (int64_t)m * e.D + n;
    const f32x4 dy = load4f(reinterpret_cast<const T*>(e.dY) + off);
    const f32x4 dS = load4f(e.dS + (int64_t)(b * e.nb + blk) * e.D + n);
    const f32x4 w = load4f(reinterpret_cast<const T*>(e.wp) + n);
    const float a = e.a[m], ds = e.ds[m];
    f32x4 o;
#pragma unroll
    for (int r = 0; r < 4; ++r) o[r] = v[r] + dy[r] + a * dS[r] + ds * w[r];
    store4(reinterpret_cast<T*>(e.dH) + off, o[0], o[1], o[2], o[3]);
  }
  __device__ __forceinline__ void apply8(int m, int n, const float (&v)[8], bool ok) const {
    if (!ok) return;
    const int b = m / e.T;
    const int t = m - b * e.T;
    const int blk = t / e.L;
    const int64_t off = (int64_t)m * e.D + n;
    float dy[8], dS[8], w[8], o[8];
    ld8(reinterpret_cast<const T*>(e.dY) + off, dy);
    ld8(e.dS + (int64_t)(b * e.nb + blk) * e.D + n, dS);
    ld8(reinterpret_cast<const T*>(e.wp) + n, w);
    const float a = e.a[m], ds = e.ds[m];
#pragma unroll
    for (int k = 0; k < 8; ++k) o[k] = v[k] + dy[k] + a * dS[k] + ds * w[k];
    st8(reinterpret_cast<T*>(e.dH) + off, o);
  }
};

// ------------------------------------------------------------------ pipelined bf16 kernel
// The bf16 path streams K slabs of 64 through a ring of STAGES LDS buffers
// with direct global->LDS loads (each 16-byte load lands at base + 16*lane
// of its instruction's 1 KB LDS window), so no register holds operand data
// on its way in and the loads of the next slabs are in flight while one is
// multiplied.
//
// LDS keeps every operand in its global orientation:
//   K-contiguous operand: [rows][64] with the 16-byte chunk c of row r
//     holding global chunk c ^ ((r / 2) % 8); a fragment is one 16-byte read.
//   M/N-contiguous operand: [64][rows] with chunk c of k-row kr holding
//     global chunk c ^ rswz(kr); a fragment is two ds_read_b64_tr_b16
//     reads.  That instruction hands lane i of each 16-lane group element
//     (i % 4) of the 4-element rows read by lanes 4j + i/4, j = 0..3; with
//     lane q addressing k-row k0 + q/4 at column c0 + 4 (q % 4), lane i
//     receives the four k values k0..k0+3 of column c0 + i, which is the
//     matrix instruction's operand layout.
// The XOR swizzles spread the 16 rows (or k-rows) a fragment read touches
// over distinct LDS banks.

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

template <int R, int BK, bool RCONTIG>
struct PipeOperand {
  static_assert(BK == 32 || BK == 64, "slab depth");
  static constexpr int ELEMS = R * BK;
  static constexpr int INSTR = ELEMS / 512;  // 1 KB per wave-wide load
  static constexpr int KCH = BK / 8;         // 16-byte chunks per K-contiguous row
  // XOR swizzle of a K-contiguous row's chunks: spreads the 16 rows of a
  // fragment read over all banks (rows are 64 or 128 bytes apart).
  __device__ __forceinline__ static int kswz(int r) {
    return BK == 64 ? ((r >> 1) & 7) : ((r >> 2) & 3);
  }
  // XOR swizzle of an M/N-contiguous k-row's chunks.  A transposing
  // fragment read has each 16-lane group read two adjacent chunks of four
  // consecutive k-rows (k-row bits 0-1; bit 2 is the second read of the
  // pair, bits 3-4 the lane group): bits 0-1 go to chunk bits 1-2, so the
  // group's eight (k-row, chunk) pairs land in eight distinct chunk slots,
  // and bit 3 ^ bit 4 to chunk bit 3, so that two groups read in the same
  // cycle use disjoint halves of the banks.  (XOR with k-row & 15 left the
  // k-row pairs 4j, 4j+1 on the same slots: a two-way bank conflict on
  // every transposing read.)
  __device__ __forceinline__ static int rswz(int kr) {
    return ((kr & 3) << 1) ^ ((kr ^ (kr >> 1)) & 8);
  }
};

// The direct loads of one operand of one workgroup.  A slab is addressed by
// a wave-uniform base pointer (scalar registers) plus a per-lane byte offset
// that does not change from slab to slab, so issuing a load costs no vector
// arithmetic.  Rows beyond the operand's last one are clamped to it (their
// products are never stored), so every address lies inside the operand; the
// buffer descriptor's size is the extent the slab may touch, so a stray
// offset would read zeros rather than leave it.
//   K-contiguous (RCONTIG false): row r of the tile, 16-byte chunk c of the
//     slab; base = P + r0 * ld + k.
//   row-contiguous (RCONTIG true): k-row kr of the slab, 16-byte chunk c of
//     the tile's rows; base = P + k * ld + c0 with c0 = min(r0, rmax - 8).
template <int R, int BK, bool RCONTIG, int NW>
struct PipeLoad {
  typedef PipeOperand<R, BK, RCONTIG> Op;
  static constexpr int PER = Op::INSTR / NW;  // loads per wave per slab
  static_assert(Op::INSTR % NW == 0, "loads per wave");
  uint32_t voff[PER];
  uint32_t extent;  // bytes a slab may touch from its base
  int r0, c0;

  __device__ __forceinline__ void setup(int row0, int rmax, int64_t ld, int wave, int lane) {
    r0 = row0;
    if constexpr (!RCONTIG) {
      constexpr int RPI = 64 / Op::KCH;  // rows per load instruction
      const int nrows = min(R, rmax - row0);
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int row = (wave * PER + i) * RPI + lane / Op::KCH;
        const int cg = (lane % Op::KCH) ^ Op::kswz(row);
        const int rr = min(row, nrows - 1);
        voff[i] = (uint32_t)(((int64_t)rr * ld + cg * 8) * 2);
      }
      extent = (uint32_t)(((int64_t)(nrows - 1) * ld + BK) * 2);
    } else {
      constexpr int CPR = R / 8;     // 16-byte chunks per k-row
      constexpr int RPI = 64 / CPR;  // k-rows per load instruction
      static_assert(CPR >= 16 && 64 % CPR == 0, "row width");
      c0 = min(row0, rmax - 8);
      const int cend = min(row0 + R, rmax);
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int kr = (wave * PER + i) * RPI + lane / CPR;
        const int cg = (lane % CPR) ^ Op::rswz(kr);
        const int gc = min(row0 + cg * 8, rmax - 8);
        voff[i] = (uint32_t)(((int64_t)kr * ld + (gc - c0)) * 2);
      }
      extent = (uint32_t)(((int64_t)(BK - 1) * ld + (cend - c0)) * 2);
    }
  }

  // Base of the slab starting at k (relative to pointer P).
  __device__ __forceinline__ const bf16* slab(const bf16* P, int64_t ld, int k) const {
    if constexpr (!RCONTIG) return P + (int64_t)r0 * ld + k;
    else return P + (int64_t)k * ld + c0;
  }

  // This wave's loads of one slab into dst (the operand's LDS region).
  // (The buffer-descriptor type exists only in the device compilation pass.)
  __device__ __forceinline__ void issue(const bf16* base, bf16* dst, int wave) const {
#if defined(__HIP_DEVICE_COMPILE__)
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, (int)extent, 0x00020000);
#pragma unroll
    for (int i = 0; i < PER; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void_t*)(dst + (wave * PER + i) * 512), 16,
                                               voff[i], 0, 0, 0);
#endif
  }

  // Fragment for rows/columns base .. base+15 of the tile, 32-wide K step ks.
  __device__ __forceinline__ static bf16x8 frag(const bf16* s, int base, int ks, int lane) {
    const int lr = lane & 15, lg = lane >> 4;
    if constexpr (!RCONTIG) {
      const int r = base + lr;
      const int c = (ks * 4 + lg) ^ Op::kswz(r);
      return lds_read_b128(s + r * BK + c * 8);
    } else {
      const int col = base + (lr & 3) * 4;
      bf16x4 h[2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int kr = ks * 32 + lg * 8 + hh * 4 + (lr >> 2);
        const int c = (col >> 3) ^ Op::rswz(kr);
        h[hh] = lds_read_tr(s + kr * R + c * 8 + (col & 7));
      }
      bf16x8 r = {h[0][0], h[0][1], h[0][2], h[0][3], h[1][0], h[1][1], h[1][2], h[1][3]};
      return r;
    }
  }
};

// Tile order.  Workgroups are dealt to the chip's 8 XCDs round-robin in
// launch order (x fastest, then y, then the split index z), and each XCD has
// its own L2.  The launch-order index is mapped so that every XCD works
// through one contiguous run of the (split, tile) sequence; within a split
// the sequence walks groups of `group` tile rows column by column.  The
// launcher picks the group height that keeps the A row panels plus B column
// panels each XCD touches smallest (xcd_group_rows), so that they are read
// from HBM once per XCD and then served from its L2.
constexpr int kXcds = 8;

__device__ __forceinline__ void xcd_tile_order(int group, int& tm, int& tn, int& z) {
  const int nx = gridDim.x, ny = gridDim.y;
  const int ntiles = nx * ny;
  const int total = ntiles * gridDim.z;
  const int bid = (blockIdx.z * ny + blockIdx.y) * nx + blockIdx.x;
  const int xcd = bid % kXcds, pos = bid / kXcds;
  const int q = total / kXcds, r = total % kXcds;
  int t = xcd < r ? xcd * (q + 1) + pos : r * (q + 1) + (xcd - r) * q + pos;
  z = t / ntiles;
  t -= z * ntiles;
  const int first = (t / (group * nx)) * group;
  const int gm = min(ny - first, group);
  const int in = t - first * nx;
  tm = first + in % gm;
  tn = in / gm;
}

// Split-K partial epilogues write the slice of their split; others ignore it.
template <class E>
__device__ __forceinline__ void bind_split(E&, int) {}

template <int BM, int BN, int BK, int STAGES, int WGM, int WGN, bool A_MC, bool B_NC, int BSEG,
          class Epi>
__global__ __launch_bounds__(WGM* WGN * 64) void gemm_pipe_kernel(int M, int N, int K,
                                                                Operand<bf16, A_MC, kSegNone> A,
                                                                Operand<bf16, B_NC, BSEG> B,
                                                                int kchunk, int group, Epi epi0) {
  constexpr int NW = WGM * WGN;
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int FM = WTM / 16, FN = WTN / 16;
  typedef PipeLoad<BM, BK, A_MC, NW> LA;
  typedef PipeLoad<BN, BK, B_NC, NW> LB;
  constexpr int AEL = LA::Op::ELEMS;
  constexpr int STAGE = AEL + LB::Op::ELEMS;
  constexpr int NI = LA::PER + LB::PER;  // loads per wave per slab
  __shared__ __attribute__((aligned(1024))) bf16 lds[STAGES * STAGE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;
  int tm, tn, z;
  xcd_tile_order(group, tm, tn, z);
  const int m0 = tm * BM, n0 = tn * BN;
  const int kbeg = z * kchunk;
  Epi epi = epi0;
  bind_split(epi, z);
  const int kend = min(K, kbeg + kchunk);
  const int nk = kend > kbeg ? (kend - kbeg) / BK : 0;

  // B split along N: the tile lies inside one part (the launcher checks that
  // the part width is a multiple of BN).
  const bf16* bptr = B.p[0];
  int bn0 = n0, bnmax = N;
  if constexpr (BSEG == kSegN) {
    const int sg = n0 / B.seg_len;
    bptr = B.p[sg];
    bn0 = n0 - sg * B.seg_len;
    bnmax = B.seg_len;
  }
  LA la;
  LB lb;
  la.setup(m0, M, A.ld, wave, lane);
  lb.setup(bn0, bnmax, B.ld, wave, lane);
  // Slab base of B at global k (B split along K: each slab lies inside one
  // part; the launcher checks that the part length is a multiple of BK).
  auto bslab = [&](int k) {
    if constexpr (BSEG == kSegK) {
      const int sg = k / B.seg_len;
      return lb.slab(B.p[sg], B.ld, k - sg * B.seg_len);
    } else {
      return lb.slab(bptr, B.ld, k);
    }
  };

  f32x4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Software pipeline: the fragments of the next 32-wide K step are read
  // from LDS while the matrix instructions of the current one run; the
  // first step of slab kt + 1 is read during the last step of slab kt,
  // right after the barrier that publishes slab kt + 1 and releases slab
  // kt's buffer for slab kt + STAGES.  Every LDS access of the loop goes
  // through inline assembly, so the waits below count all of them.
  constexpr int NKS = BK / 32;  // K steps per slab
  static_assert(NKS == 1 || NKS == 2, "slab depth");
  constexpr int UNR = NKS == 1 ? 2 : 1;  // slabs per trip, so that fragment sets alternate
  constexpr int NR = FM * (A_MC ? 2 : 1) + FN * (B_NC ? 2 : 1);  // LDS reads per K step
  constexpr int NRW = NR < 15 ? NR : 15;
  bf16x8 fa[2][FM], fb[2][FN];
  auto read_step = [&](const bf16* s, int ks, bf16x8(&a)[FM], bf16x8(&b)[FN]) {
#pragma unroll
    for (int i = 0; i < FM; ++i) a[i] = LA::frag(s, wm * WTM + i * 16, ks, lane);
#pragma unroll
    for (int j = 0; j < FN; ++j) b[j] = LB::frag(s + AEL, wn * WTN + j * 16, ks, lane);
  };
  // The matrix instructions are inline assembly too, so that they stay
  // between the reads and waits that feed them (the accumulators stay put in
  // AGPRs).  The compiler's hazard tracking does not see them: s_nop 2
  // covers a vector write of an operand just before, and the loop's end
  // waits out their passes before anything reads the accumulators.
  auto mma_step = [&](bf16x8(&a)[FM], bf16x8(&b)[FN]) {
    asm volatile("s_nop 2");
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0"
                     : "+a"(acc[i][j])
                     : "v"(b[j]), "v"(a[i]));
  };
  // Waits until slab `need` has landed, given that slabs up to `last` were
  // issued (each wave's own loads; the barrier that follows covers the rest).
  auto wait_slab = [&](int need, int last) {
    const int after = last - need;
    if (after >= 4 && STAGES >= 5) wait_vmcnt<4 * NI>();
    else if (after >= 3 && STAGES >= 4) wait_vmcnt<3 * NI>();
    else if (after >= 2 && STAGES >= 3) wait_vmcnt<2 * NI>();
    else if (after >= 1) wait_vmcnt<NI>();
    else wait_vmcnt<0>();
  };
  auto buf = [&](int kt) { return lds + (kt % STAGES) * STAGE; };

  // Prologue: every buffer of the ring receives its slab.
#pragma unroll
  for (int st = 0; st < STAGES; ++st) {
    if (st < nk) {
      bf16* sa = lds + st * STAGE;
      const int k = kbeg + st * BK;
      la.issue(la.slab(A.p[0], A.ld, k), sa, wave);
      lb.issue(bslab(k), sa + AEL, wave);
    }
  }
  if (nk > 0) {
    wait_slab(0, min(nk, STAGES) - 1);
    __builtin_amdgcn_s_barrier();
    read_step(lds, 0, fa[0], fb[0]);
  }

  for (int kt0 = 0; kt0 < nk; kt0 += UNR) {
#pragma unroll
    for (int uu = 0; uu < UNR; ++uu) {
      const int kt = kt0 + uu;
      if (UNR > 1 && kt >= nk) break;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const int c = (uu * NKS + ks) & 1;  // fragment set of this step
        if (ks + 1 < NKS) {
          read_step(buf(kt), ks + 1, fa[c ^ 1], fb[c ^ 1]);
          lds_wait<NRW>();  // this step's fragments have landed
        } else {
          lds_wait<0>();  // this step's too, and this wave is done reading slab kt
          if (kt + 1 < nk) {
            wait_slab(kt + 1, min(nk, kt + STAGES) - 1);
            // Slab kt + 1 is visible to all waves, and no wave reads slab kt
            // any more: its buffer takes slab kt + STAGES.
            __builtin_amdgcn_s_barrier();
            const int nxt = kt + STAGES;
            if (nxt < nk) {
              bf16* sn = buf(kt);
              const int k = kbeg + nxt * BK;
              la.issue(la.slab(A.p[0], A.ld, k), sn, wave);
              lb.issue(bslab(k), sn + AEL, wave);
            }
            read_step(buf(kt + 1), 0, fa[c ^ 1], fb[c ^ 1]);
          }
        }
        mma_step(fa[c], fb[c]);
      }
    }
  }
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7");

  static_assert(STAGES * STAGE * 2 >= BM * BN * 4, "staging tile fits the LDS ring");
  staged_epilogue<BM, BN, FM, FN, WTM, WTN, NW * 64>(epi, acc, reinterpret_cast<float*>(lds), m0,
                                                      n0, wm, wn, M, N, tid);
}

// The tied head of the language model, logits z = f E^T, consumed tile by
// tile and never stored.  EpiHeadStats leaves, for every row of a 128-column
// tile, (max, sum of exp(z - max)) over the columns below V at
// part[2 (m ntile + tile)]; the staged epilogue hands a row's 128 columns to
// 16 consecutive threads (one DPP row), which reduce them together.
// EpiHeadGrad stores the loss gradient (softmax - onehot) * inv_n, zero in
// the padding columns, given each row's log-sum-exp.
constexpr float kLog2e = 1.4426950408889634f;
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp_mov<0xB1>(v));
  v = fmaxf(v, dpp_mov<0x4E>(v));
  v = fmaxf(v, dpp_mov<0x141>(v));
  return fmaxf(v, dpp_mov<0x140>(v));
}
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_mov<0xB1>(v);
  v += dpp_mov<0x4E>(v);
  v += dpp_mov<0x141>(v);
  return v + dpp_mov<0x140>(v);
}
struct EpiHeadStats {
  float* part;
  int ntile;
  int V;
  __device__ __forceinline__ void apply8(int m, int n, const float (&v)[8], bool ok) const {
    // every thread takes part (the DPP steps read neighbours); only the
    // row's first thread stores
    float mx = -INFINITY;
#pragma unroll
    for (int e = 0; e < 8; ++e) mx = fmaxf(mx, n + e < V ? v[e] : -INFINITY);
    mx = row16_max(mx);
    const float ml = mx == -INFINITY ? 0.f : mx * kLog2e;
    float sum = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float x = exp2_fast(fmaf(v[e], kLog2e, -ml));
      sum += n + e < V ? x : 0.f;
    }
    sum = row16_sum(sum);
    if (ok && (n & 127) == 0) {
      float* q = part + 2 * ((int64_t)m * ntile + (n >> 7));
      q[0] = mx;
      q[1] = sum;
    }
  }
};
struct EpiHeadGrad {
  bf16* G;
  int64_t ld;
  const float* lse;
  const int32_t* tgt;
  int V;
  float inv_n;
  __device__ __forceinline__ void apply8(int m, int n, const float (&v)[8], bool ok) const {
    if (!ok) return;
    const float ll = lse[m] * kLog2e;
    const int tk = min(max(tgt[m], 0), V - 1);
    float o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int c = n + e;
      float p = c < V ? exp2_fast(fmaf(v[e], kLog2e, -ll)) : 0.f;
      if (c == tk) p -= 1.f;
      o[e] = p * inv_n;
    }
    st8(G + (int64_t)m * ld + n, o);
  }
};

// ------------------------------------------------------------------ launch

// Tile rows plus tile columns (counted per split, whose K ranges differ)
// that the tiles [a, b) of the (split, tile) sequence touch with group
// height g.
int64_t panels_touched(int64_t a, int64_t b, int g, int nx, int ny) {
  const int64_t ntiles = (int64_t)nx * ny;
  int64_t cost = 0;
  while (a < b) {  // one split at a time
    const int64_t z = a / ntiles, ts = a - z * ntiles;
    const int64_t te = std::min(b, (z + 1) * ntiles) - z * ntiles;
    int64_t cols = 0;
    for (int64_t gi = ts / ((int64_t)g * nx); gi * g * nx < te; ++gi) {
      const int64_t first = gi * g, hg = std::min<int64_t>(g, ny - first);
      const int64_t gs = first * nx;
      const int64_t la = std::max(ts, gs) - gs, lb = std::min(te, gs + hg * nx) - gs;
      if (lb <= la) continue;
      cost += std::min(hg, lb - la);
      cols += (lb - 1) / hg - la / hg + 1;
    }
    cost += std::min<int64_t>(cols, nx);
    a = (z + 1) * ntiles;
  }
  return cost;
}

// Group height for xcd_tile_order.  A candidate costs, for the worst XCD,
// the panels its whole run touches (each read from HBM into that XCD's L2
// once) plus the panels its first 64 tiles touch (roughly what it holds at
// once: two workgroups on each of its 32 CUs), which must fit its L2
// together with the output being written.  The cheapest candidate wins,
// the smallest on ties.
int xcd_group_rows_search(int nx, int ny, int nz) {
  const int64_t total = (int64_t)nx * ny * nz;
  const int64_t q = total / kXcds, r = total % kXcds;
  int best = 1;
  int64_t best_cost = -1;
  for (int g = 1; g <= ny && g <= 256; ++g) {
    int64_t worst = 0;
    for (int x = 0; x < kXcds; ++x) {
      const int64_t a = x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q;
      const int64_t b = a + q + (x < r ? 1 : 0);
      const int64_t cost = panels_touched(a, b, g, nx, ny) +
                           panels_touched(a, std::min<int64_t>(b, a + 64), g, nx, ny);
      worst = std::max(worst, cost);
    }
    if (best_cost < 0 || worst < best_cost) {
      best_cost = worst;
      best = g;
    }
  }
  return best;
}

// The search above, remembered per grid shape (a layer launches the same
// few shapes over and over; one small table per host thread).
int xcd_group_rows(int nx, int ny, int nz) {
  struct Entry { int nx, ny, nz, g; };
  thread_local Entry cache[16];
  thread_local int used = 0;
  for (int i = 0; i < used && i < 16; ++i)
    if (cache[i].nx == nx && cache[i].ny == ny && cache[i].nz == nz) return cache[i].g;
  const int g = xcd_group_rows_search(nx, ny, nz);
  cache[used % 16] = Entry{nx, ny, nz, g};
  ++used;
  return g;
}

template <typename T, bool AMC, bool BNC, int SEG, class Epi>
hipError_t launch(const GemmDesc& g, const Epi& epi, hipStream_t s) {
  constexpr int BK = KSlab<T>::BK;
  Operand<T, AMC, kSegNone> A{{(const T*)g.A, nullptr, nullptr}, g.lda, 0};
  Operand<T, BNC, SEG> B{{(const T*)g.B[0], (const T*)g.B[1], (const T*)g.B[2]}, g.ldb,
                         g.seg_len};
  int splits = g.splits < 1 ? 1 : g.splits;
  int kchunk = (g.K + splits - 1) / splits;
  kchunk = (kchunk + BK - 1) / BK * BK;
  if (kchunk < BK) kchunk = BK;
  if (g.kchunk > 0) kchunk = g.kchunk;
  splits = (g.K + kchunk - 1) / kchunk;
  if (splits < 1) splits = 1;
  dim3 grid((g.N + BN - 1) / BN, (g.M + BM - 1) / BM, splits);
  hipLaunchKernelGGL((gemm_kernel<T, AMC, BNC, SEG, Epi>), grid, dim3(kThreads), 0, s, g.M, g.N,
                     g.K, A, B, kchunk, epi);
  return hipGetLastError();
}

// Pipelined bf16 launch: 128 x 128 tiles, two 32 KB slabs in flight, so
// that two workgroups share a CU (measured faster on these shapes than a
// deeper ring with one workgroup per CU).  Eight waves of 64 x 32 by
// default: more waves to cover the load and LDS latencies, at 1.5x the
// fragment reads per matrix instruction.  Four waves of 64 x 64 stay on
// the weight gradients whose operands are both read transposed and that
// fill the chip with splits, and on products whose B is split along K (the
// input gradient of Q, K, V): there eight waves measured slower.  The
// layer's forward + backward step took 308 instead of 316 us.  Needs the K
// range of every split to be a whole number of 64-wide slabs.
template <int WGM, int WGN, bool AMC, bool BNC, int SEG, class Epi>
hipError_t launch_pipe_w(const GemmDesc& g, const Epi& epi, hipStream_t s) {
  constexpr int PBM = 128, PBN = 128, PBK = 64, ST = 2;
  Operand<bf16, AMC, kSegNone> A{{(const bf16*)g.A, nullptr, nullptr}, g.lda, 0};
  Operand<bf16, BNC, SEG> B{{(const bf16*)g.B[0], (const bf16*)g.B[1], (const bf16*)g.B[2]}, g.ldb,
                            g.seg_len};
  int splits = g.splits < 1 ? 1 : g.splits;
  int kchunk = (g.K + splits - 1) / splits;
  kchunk = (kchunk + 63) / 64 * 64;
  if (g.kchunk > 0) kchunk = g.kchunk;
  splits = (g.K + kchunk - 1) / kchunk;
  dim3 grid((g.N + PBN - 1) / PBN, (g.M + PBM - 1) / PBM, splits);
  const int group = xcd_group_rows((int)grid.x, (int)grid.y, (int)grid.z);
  hipLaunchKernelGGL((gemm_pipe_kernel<PBM, PBN, PBK, ST, WGM, WGN, AMC, BNC, SEG, Epi>), grid,
                     dim3(WGM * WGN * 64), 0, s, g.M, g.N, g.K, A, B, kchunk, group, epi);
  return hipGetLastError();
}

template <bool AMC, bool BNC, int SEG, class Epi>
hipError_t launch_pipe(const GemmDesc& g, const Epi& epi, hipStream_t s) {
  if constexpr (AMC) {
    int splits = g.splits < 1 ? 1 : g.splits;
    if (g.kchunk > 0) splits = (g.K + g.kchunk - 1) / g.kchunk;
    const int64_t wgs = (int64_t)((g.N + 127) / 128) * ((g.M + 127) / 128) * splits;
    if (wgs >= 256) return launch_pipe_w<2, 2, AMC, BNC, SEG>(g, epi, s);
  }
  if constexpr (SEG == kSegK) return launch_pipe_w<2, 2, AMC, BNC, SEG>(g, epi, s);
  return launch_pipe_w<2, 4, AMC, BNC, SEG>(g, epi, s);
}

template <typename T, bool AMC, bool BNC, int SEG, class Epi>
hipError_t launch_any(const GemmDesc& g, const Epi& epi, hipStream_t s) {
  if constexpr (sizeof(T) == 2) {
    // The pipelined kernel needs whole 64-deep slabs, operands of at least
    // 8 rows, and B parts that never split a tile (N) or a slab (K).
    bool ok = g.K % 64 == 0 && g.M >= 8 && g.N >= 8;
    if (SEG == kSegN) ok = ok && g.seg_len % 128 == 0;
    if (SEG == kSegK) ok = ok && g.seg_len % 64 == 0;
    if (ok) return launch_pipe<AMC, BNC, SEG>(g, epi, s);
  }
  return launch<T, AMC, BNC, SEG>(g, epi, s);
}

template <typename T, class Epi>
hipError_t dispatch_store(const GemmDesc& g, const Epi& epi, hipStream_t s) {
  if (!g.a_mcontig && g.b_ncontig && g.seg == kSegNone) return launch_any<T, false, true, kSegNone>(g, epi, s);
  if (!g.a_mcontig && g.b_ncontig && g.seg == kSegN) return launch_any<T, false, true, kSegN>(g, epi, s);
  if (!g.a_mcontig && !g.b_ncontig && g.seg == kSegNone) return launch_any<T, false, false, kSegNone>(g, epi, s);
  if (!g.a_mcontig && !g.b_ncontig && g.seg == kSegK) return launch_any<T, false, false, kSegK>(g, epi, s);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t gemm_store(DType dt, const GemmDesc& g, void* C, int64_t ldc, bool c_f32,
                      const void* add, int64_t ld_add, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (dt == DType::BF16) {
    if (c_f32) return dispatch_store<bf16>(g, EpiStore<float, bf16>{(float*)C, ldc, (const bf16*)add, ld_add}, s);
    return dispatch_store<bf16>(g, EpiStore<bf16, bf16>{(bf16*)C, ldc, (const bf16*)add, ld_add}, s);
  }
  return dispatch_store<float>(g, EpiStore<float, float>{(float*)C, ldc, (const float*)add, ld_add}, s);
}

namespace {

// Split-K plan: at most two workgroups per CU of 128 x 128 tiles (two fit in
// LDS at once), so that the whole grid is resident in one round; every split
// at least min_k deep in K (rounded to a multiple of 64).  Returns the number
// of splits; *kchunk is the K range of each.
static int splitk_plan(int M, int N, int K, int min_k, int* kchunk) {
  const int tiles = ((M + 127) / 128) * ((N + 127) / 128);
  int sp = 512 / tiles;
  const int kmax = K / min_k;
  if (sp > kmax) sp = kmax;
  if (sp < 1) sp = 1;
  int kc = (K + sp - 1) / sp;
  kc = (kc + 63) / 64 * 64;
  *kchunk = kc;
  return (K + kc - 1) / kc;
}

// Writes (or accumulates into) up to three float32 outputs split along N.
struct EpiSegOut {
  float* C[3];
  int64_t ldc;
  int seg;
  int accumulate;
  __device__ __forceinline__ void operator()(int m, int n, f32x4 v) const {
    const int sg = n / seg;
    float* base = C[sg];
    if (!base) return;
    f32x4* dst = reinterpret_cast<f32x4*>(base + (int64_t)m * ldc + (n - sg * seg));
    if (accumulate) v += *dst;
    *dst = v;
  }
  // (Output segments are multiples of 8 columns wide, so 8 columns never
  // straddle two of them.)
  __device__ __forceinline__ void apply8(int m, int n, const float (&v)[8], bool ok) const {
    if (!ok) return;
    const int sg = n / seg;
    float* base = C[sg];
    if (!base) return;
    float* dst = base + (int64_t)m * ldc + (n - sg * seg);
    float o[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) o[k] = v[k];
    if (accumulate) {
      float a[8];
      ld8(dst, a);
#pragma unroll
      for (int k = 0; k < 8; ++k) o[k] += a[k];
    }
    st8(dst, o);
  }
};

template <typename T, class Epi>
hipError_t dispatch_any(const GemmDesc& g, const Epi& epi, hipStream_t s) {
  if (g.seg == kSegK) {  // B split along K (K-contiguous B only): bf16 products
    if constexpr (sizeof(T) == 2) {
      if (!g.a_mcontig && !g.b_ncontig) return launch_any<T, false, false, kSegK>(g, epi, s);
    }
    return hipErrorInvalidValue;
  }
  if (g.a_mcontig && g.b_ncontig && g.seg == kSegNone) return launch_any<T, true, true, kSegNone>(g, epi, s);
  if (!g.a_mcontig && g.b_ncontig && g.seg == kSegNone) return launch_any<T, false, true, kSegNone>(g, epi, s);
  if (!g.a_mcontig && !g.b_ncontig && g.seg == kSegNone) return launch_any<T, false, false, kSegNone>(g, epi, s);
  return hipErrorInvalidValue;
}

}  // namespace

int gemm_splitk_splits(int M, int N, int K, int min_k) {
  int kc;
  return splitk_plan(M, N, K, min_k, &kc);
}

size_t gemm_splitk_partial_bytes(int M, int N, int K, int min_k) {
  int kc;
  const int sp = splitk_plan(M, N, K, min_k, &kc);
  return sp > 1 ? (size_t)sp * M * N * sizeof(float) : 0;
}

size_t gemm_wgrad_partial_bytes(int M, int N, int K) {
  return gemm_splitk_partial_bytes(M, N, K, 512);
}

hipError_t gemm_splitk_product(DType dt, const GemmDesc& g0, float* partial, float* C0, float* C1,
                               float* C2, int64_t ldc, int seg_len_n, bool accumulate, int min_k,
                               int* splits, hipStream_t s) {
  *splits = 0;
  if (g0.M <= 0 || g0.N <= 0) return hipSuccess;
  if (g0.N % 8 != 0 || seg_len_n % 8 != 0) return hipErrorInvalidValue;
  if (g0.seg == kSegN || (g0.seg == kSegK && (g0.b_ncontig || g0.a_mcontig)))
    return hipErrorInvalidValue;
  GemmDesc g = g0;
  int kc;
  g.splits = splitk_plan(g.M, g.N, g.K, min_k, &kc);
  g.kchunk = kc;  // exactly g.splits slices of `partial` get written
  *splits = g.splits;
  if (g.splits == 1) {
    EpiSegOut e{{C0, C1, C2}, ldc, seg_len_n, accumulate ? 1 : 0};
    return dt == DType::BF16 ? dispatch_any<bf16>(g, e, s) : dispatch_any<float>(g, e, s);
  }
  EpiPartial e{partial, g.N, (int64_t)g.M * g.N};
  return dt == DType::BF16 ? dispatch_any<bf16>(g, e, s) : dispatch_any<float>(g, e, s);
}

hipError_t gemm_splitk_reduce(const float* partial, int splits, int M, int N, float* C0, float* C1,
                              float* C2, int64_t ldc, int seg_len_n, bool accumulate,
                              hipStream_t s) {
  if (splits <= 1 || M <= 0 || N <= 0) return hipSuccess;
  const int64_t total = (int64_t)M * N / 4;
  const int64_t blocks = (total + 63) / 64;
  hipLaunchKernelGGL(wgrad_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, s, partial, splits,
                     M, N, C0, C1, C2, ldc, seg_len_n, accumulate ? 1 : 0);
  return hipGetLastError();
}

hipError_t gemm_splitk(DType dt, const GemmDesc& g, float* partial, float* C0, float* C1,
                       float* C2, int64_t ldc, int seg_len_n, bool accumulate, int min_k,
                       hipStream_t s) {
  int sp = 0;
  hipError_t e = gemm_splitk_product(dt, g, partial, C0, C1, C2, ldc, seg_len_n, accumulate, min_k,
                                     &sp, s);
  if (e != hipSuccess) return e;
  return gemm_splitk_reduce(partial, sp, g.M, g.N, C0, C1, C2, ldc, seg_len_n, accumulate, s);
}

hipError_t gemm_wgrad(DType dt, const GemmDesc& g, float* partial, float* C0, float* C1,
                      float* C2, int64_t ldc, int seg_len_n, bool accumulate, hipStream_t s) {
  if (!(g.a_mcontig && g.b_ncontig && g.seg == kSegNone)) return hipErrorInvalidValue;
  return gemm_splitk(dt, g, partial, C0, C1, C2, ldc, seg_len_n, accumulate, 512, s);
}

hipError_t gemm_score(DType dt, const GemmDesc& g, void* C, const void* wp, float* sp,
                      hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (g.N % 64 != 0 || !(!g.a_mcontig && g.b_ncontig && g.seg == kSegNone))
    return hipErrorInvalidValue;
  if (dt == DType::BF16)
    return launch_any<bf16, false, true, kSegNone>(
        g, EpiScore<bf16>{(bf16*)C, g.N, (const bf16*)wp, sp, g.N / 64}, s);
  return launch<float, false, true, kSegNone>(
      g, EpiScore<float>{(float*)C, g.N, (const float*)wp, sp, g.N / 64}, s);
}

hipError_t gemm_gate(DType dt, const GemmDesc& g, const GateEpi& e, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (!(!g.a_mcontig && g.b_ncontig && g.seg == kSegNone)) return hipErrorInvalidValue;
  if (dt == DType::BF16) return launch_any<bf16, false, true, kSegNone>(g, EpiGate<bf16>{e}, s);
  return launch<float, false, true, kSegNone>(g, EpiGate<float>{e}, s);
}

hipError_t gemm_gelu(DType dt, const GemmDesc& g, void* U, void* A, int64_t ld, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (dt != DType::BF16 || g.a_mcontig || g.seg != kSegNone) return hipErrorInvalidValue;
  const EpiGelu<bf16> e{(bf16*)U, (bf16*)A, ld};
  if (g.b_ncontig) return launch_any<bf16, false, true, kSegNone>(g, e, s);
  return launch_any<bf16, false, false, kSegNone>(g, e, s);
}

hipError_t gemm_gelu_bwd(DType dt, const GemmDesc& g, const void* U, void* dU, int64_t ld,
                         hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (dt != DType::BF16 || g.a_mcontig || g.seg != kSegNone) return hipErrorInvalidValue;
  const EpiGeluBwd<bf16> e{(const bf16*)U, (bf16*)dU, ld};
  if (g.b_ncontig) return launch_any<bf16, false, true, kSegNone>(g, e, s);
  return launch_any<bf16, false, false, kSegNone>(g, e, s);
}

// Both head products need the pipelined kernel (its epilogue layout) and
// whole 128-column tiles.
static bool head_shape_ok(const GemmDesc& g) {
  return !g.a_mcontig && !g.b_ncontig && g.seg == kSegNone && g.splits <= 1 && g.K % 64 == 0 &&
         g.M >= 8 && g.N % 128 == 0;
}

hipError_t gemm_head_stats(const GemmDesc& g, float* part, int V, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (!head_shape_ok(g) || V < 1 || V > g.N) return hipErrorInvalidValue;
  return launch_pipe<false, false, kSegNone>(g, EpiHeadStats{part, g.N / 128, V}, s);
}

hipError_t gemm_head_grad(const GemmDesc& g, void* G, int64_t ld, const float* lse,
                          const int32_t* tgt, int V, float inv_n, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (!head_shape_ok(g) || V < 1 || V > g.N) return hipErrorInvalidValue;
  return launch_pipe<false, false, kSegNone>(g, EpiHeadGrad{(bf16*)G, ld, lse, tgt, V, inv_n}, s);
}

hipError_t gemm_hbar(DType dt, const GemmDesc& g, const HbarEpi& e, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (!(!g.a_mcontig && !g.b_ncontig && g.seg == kSegNone)) return hipErrorInvalidValue;
  if (dt == DType::BF16) return launch_any<bf16, false, false, kSegNone>(g, EpiHbar<bf16>{e}, s);
  return launch<float, false, false, kSegNone>(g, EpiHbar<float>{e}, s);
}

}  // namespace bcmt
