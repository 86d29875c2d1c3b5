// Tiled matrix product on the CDNA4 matrix cores, with fused epilogues.
//
// Serves every dense projection of the layer (Sec. 3.3 Q/K/V and W_O,
// Sec. 3.5 W_m, Sec. 3.8 W_g) and their backward products.
//
// Workgroup tile 128 x 128, four waves in a 2 x 2 grid, each wave 64 x 64 as
// 4 x 4 sub-tiles of 16 x 16.  The K loop stages one BK-wide slab of both
// operands in LDS, double buffered: the next slab's global loads are issued
// before the current slab's matrix instructions and written to the other LDS
// buffer afterwards, so one barrier per slab suffices.
//
// LDS holds both operands "K-contiguous" (row = m or n, 8 consecutive k per
// 16-byte read), which is what a lane feeds the matrix instruction.  An
// operand stored with M/N contiguous in memory is transposed on the way in:
// a thread loads an 8 x 8 (bf16) or 4 x 4 (f32) sub-block as 16-byte rows and
// writes it back transposed, 16 bytes per row.
//
// The matrix instruction is issued with the B tile as its first operand, so
// a lane ends up holding four consecutive output columns of one output row:
// the epilogue stores 8 (bf16) or 16 (f32) contiguous bytes per lane.
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
                                                        Epi epi) {
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

#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + wm * 64 + i * 16 + lr;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + wn * 64 + j * 16 + lg * 4;
      if (m < M && n < N) epi(m, n, acc[i][j]);
    }
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
};

struct EpiAtomic {
  float* C[3];
  int64_t ldc;
  int seg;
  __device__ __forceinline__ void operator()(int m, int n, f32x4 v) const {
    const int s = n / seg;
    float* base = C[s];
    if (!base) return;
    float* p = base + (int64_t)m * ldc + (n - s * seg);
#pragma unroll
    for (int r = 0; r < 4; ++r) unsafeAtomicAdd(p + r, v[r]);
  }
};

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
    f32x4 x = {0.f, 0.f, 0.f, 0.f};
    if (e.X) x = load4f(reinterpret_cast<const T*>(e.X) + off);
    f32x4 g, y;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      g[r] = sigmoidf_(u[r]);
      y[r] = h[r] + g[r] * c[r] + x[r];
    }
    store4(reinterpret_cast<T*>(e.Y) + off, y[0], y[1], y[2], y[3]);
    store4(reinterpret_cast<T*>(e.G) + off, g[0], g[1], g[2], g[3]);
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
};

// ------------------------------------------------------------------ launch

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
  splits = (g.K + kchunk - 1) / kchunk;
  if (splits < 1) splits = 1;
  dim3 grid((g.N + BN - 1) / BN, (g.M + BM - 1) / BM, splits);
  hipLaunchKernelGGL((gemm_kernel<T, AMC, BNC, SEG, Epi>), grid, dim3(kThreads), 0, s, g.M, g.N,
                     g.K, A, B, kchunk, epi);
  return hipGetLastError();
}

template <typename T, class Epi>
hipError_t dispatch_store(const GemmDesc& g, const Epi& epi, hipStream_t s) {
  if (!g.a_mcontig && g.b_ncontig && g.seg == kSegNone) return launch<T, false, true, kSegNone>(g, epi, s);
  if (!g.a_mcontig && g.b_ncontig && g.seg == kSegN) return launch<T, false, true, kSegN>(g, epi, s);
  if (!g.a_mcontig && !g.b_ncontig && g.seg == kSegNone) return launch<T, false, false, kSegNone>(g, epi, s);
  if (!g.a_mcontig && !g.b_ncontig && g.seg == kSegK) return launch<T, false, false, kSegK>(g, epi, s);
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

hipError_t gemm_atomic(DType dt, const GemmDesc& g, float* C0, float* C1, float* C2, int64_t ldc,
                       int seg_len_n, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0 || g.K <= 0) return hipSuccess;
  if (!(g.a_mcontig && g.b_ncontig && g.seg == kSegNone)) return hipErrorInvalidValue;
  EpiAtomic e{{C0, C1, C2}, ldc, seg_len_n};
  if (dt == DType::BF16) return launch<bf16, true, true, kSegNone>(g, e, s);
  return launch<float, true, true, kSegNone>(g, e, s);
}

hipError_t gemm_gate(DType dt, const GemmDesc& g, const GateEpi& e, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (!(!g.a_mcontig && g.b_ncontig && g.seg == kSegNone)) return hipErrorInvalidValue;
  if (dt == DType::BF16) return launch<bf16, false, true, kSegNone>(g, EpiGate<bf16>{e}, s);
  return launch<float, false, true, kSegNone>(g, EpiGate<float>{e}, s);
}

hipError_t gemm_hbar(DType dt, const GemmDesc& g, const HbarEpi& e, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  if (!(!g.a_mcontig && !g.b_ncontig && g.seg == kSegNone)) return hipErrorInvalidValue;
  if (dt == DType::BF16) return launch<bf16, false, false, kSegNone>(g, EpiHbar<bf16>{e}, s);
  return launch<float, false, false, kSegNone>(g, EpiHbar<float>{e}, s);
}

}  // namespace bcmt
