// The memory path of the layer: adaptive block summaries (Sec. 3.4), the
// normalised exponential causal memory (Sec. 3.5) and the bandwidth-bound
// parts of the backward pass.
//
// All of these stream [B, T, D] activations once and keep block-level
// quantities ([B, N_b, D], float32) tiny, so they are written for coalesced
// 16-byte row accesses and wave-level reductions, not for the matrix cores.
//
// Decay recurrences.  With Z_i = sum_{j<=i} g^(i-j) and N_i = sum_{j<=i}
// g^(i-j) S_j (0-based blocks), the memory is M_i = N_i / Z_i and
//   N_i = g N_{i-1} + S_i,  Z_i = g Z_{i-1} + 1.
// One workgroup owns 32 feature columns of one batch element over all
// blocks, so no workgroup ever waits on another.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace bcmt {
namespace {

// The pooling backward uses one workgroup per chunk of a block's tokens: up
// to 16 waves, each wave taking TB whole rows at a time (their rows are
// loaded together, then reduced together), so that enough loads are in
// flight per CU.

// Tokens a wave loads at once for rows of NVJ 16-byte vectors per lane.
template <int NVJ> struct TokBatch { static constexpr int TB = NVJ >= 4 ? 2 : (NVJ == 2 ? 4 : 8); };

__device__ __forceinline__ float block_reduce_sum(float v, float* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float s = 0.f;
  const int nw = blockDim.x >> 6;
  for (int w = 0; w < nw; ++w) s += red[w];
  return s;
}

// ------------------------------------------------------------------ column-chunk layout
// Pooling (forward) and the gate backward walk a block's tokens over a chunk
// of columns: workgroup = (block, batch element, chunk of 16 vectors of
// 16 bytes), thread = (vector v, token group tg) with 16 of each; thread
// (v, tg) visits tokens bs + tg, bs + tg + 16, ... and the 16 token groups
// are merged in LDS.  No reduction crosses workgroups, and a launch has
// N_b * B * ceil(D / chunk) workgroups.
constexpr int kVec = 16, kTg = 16;

// ------------------------------------------------------------------ pooling (forward)
// s_t = H[t] . w_p arrives as np partial sums per token (written by the
// output projection's epilogue); a = softmax of s over the block;
// S_i = sum_t a_t H[t].  The block's tokens are taken 256 at a time: their
// scores go to LDS (one token per thread) with the tile's max and
// exponential sum, then every thread adds its tokens' weighted rows with the
// loads of eight tokens in flight; the running max is the same for the whole
// workgroup, so only the token groups' sums remain to be added at the end.
// Chunk 0 of each block also writes s (for the backward) and the block's
// softmax statistics (max, normaliser); S_i is written in float32 and in
// the compute type (the operand of the memory projection).
__device__ __forceinline__ float block_max256(float v, float* red) {
  v = wave_max(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) red[wave] = v;
  __syncthreads();
  const float r = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  return r;
}
__device__ __forceinline__ float block_sum256(float v, float* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) red[wave] = v;
  __syncthreads();
  const float r = (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  return r;
}

// A token's score from its np partial sums, added in order; the loads are
// issued sixteen at a time, so that their latencies overlap.
__device__ __forceinline__ float score_sum(const float* __restrict__ q, int np) {
  float x = 0.f;
  for (int k0 = 0; k0 < np; k0 += 16) {
    float t[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) t[u] = k0 + u < np ? q[k0 + u] : 0.f;
#pragma unroll
    for (int u = 0; u < 16; ++u) x += t[u];
  }
  return x;
}

// Clears zero[0 .. n) as a side task shared by every workgroup of a launch
// (the records of a later kernel on the same stream).
__device__ __forceinline__ void clear_share(float* zero, int64_t n) {
  if (!zero) return;
  const int64_t G = (int64_t)gridDim.x * gridDim.y * gridDim.z;
  const int64_t g = ((int64_t)blockIdx.z * gridDim.y + blockIdx.y) * gridDim.x + blockIdx.x;
  const int64_t per = (n + G - 1) / G;
  const int64_t e = min(n, (g + 1) * per);
  for (int64_t k = g * per + threadIdx.x; k < e; k += blockDim.x) zero[k] = 0.f;
}

template <typename T>
__global__ __launch_bounds__(256) void pool_fwd_kernel(const T* __restrict__ H,
                                                       const float* __restrict__ sp, int np,
                                                       float* __restrict__ s_out,
                                                       float* __restrict__ S, T* __restrict__ St,
                                                       float* __restrict__ stats, int Tn, int D,
                                                       int L, int nb, float* __restrict__ zero,
                                                       int64_t nzero) {
  constexpr int VE = Vec16<T>::N;
  constexpr int U = 8;
  typedef typename Vec16<T>::type vec;
  clear_share(zero, nzero);
  __shared__ float racc[kTg][kVec * VE];
  __shared__ float sc[256];
  __shared__ float red[4];
  const int tid = threadIdx.x;
  const int v = tid % kVec, tg = tid / kVec;
  const int i = blockIdx.x, b = blockIdx.y;
  const int c0 = blockIdx.z * kVec * VE;
  const int col = c0 + v * VE;
  const bool act = col < D;
  const int bs = i * L;
  const int be = min(bs + L, Tn);
  const bool first = blockIdx.z == 0;
  const T* hb = H + (int64_t)b * Tn * D + col;

  float m = -INFINITY, l = 0.f, acc[VE];
#pragma unroll
  for (int e = 0; e < VE; ++e) acc[e] = 0.f;
  for (int t0 = bs; t0 < be; t0 += 256) {
    const int n = min(256, be - t0);
    float x = -INFINITY;
    if (tid < n) {
      const int64_t row = (int64_t)b * Tn + t0 + tid;
      x = score_sum(sp + row * np, np);
      if (first) s_out[row] = x;
    }
    sc[tid] = x;
    const float mn = fmaxf(m, block_max256(x, red));  // also publishes sc[]
    const float f = __expf(m - mn);
    l = l * f + block_sum256(tid < n ? __expf(x - mn) : 0.f, red);
#pragma unroll
    for (int e = 0; e < VE; ++e) acc[e] *= f;
    m = mn;
    if (act) {
      for (int k0 = tg; k0 < n; k0 += U * kTg) {
        vec h[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int k = k0 + u * kTg;
          h[u] = k < n ? load16(hb + (int64_t)(t0 + k) * D) : vec{};
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int k = k0 + u * kTg;
          const float w = k < n ? __expf(sc[k] - mn) : 0.f;
#pragma unroll
          for (int e = 0; e < VE; ++e) acc[e] += w * to_f32(h[u][e]);
        }
      }
    }
    __syncthreads();  // sc[] is rewritten by the next tile
  }
#pragma unroll
  for (int e = 0; e < VE; ++e) racc[tg][v * VE + e] = acc[e];
  __syncthreads();
  const float inv = 1.0f / l;
  const int64_t brow = (int64_t)(b * nb + i);
  if (tid < kVec * VE && c0 + tid < D) {
    float sum = 0.f;
    for (int k = 0; k < kTg; ++k) sum += racc[k][tid];
    S[brow * D + c0 + tid] = sum * inv;
    St[brow * D + c0 + tid] = from_f32<T>(sum * inv);
  }
  if (first && tid == 0) {
    stats[brow * 2] = m;
    stats[brow * 2 + 1] = l;
  }
}

// Whole-row pooling: one workgroup per (block, batch element) over all D
// columns, used when there are enough such pairs to fill the chip.  Thread
// = (16-byte vector v of the row, token group tg); the block's scores are
// formed once per workgroup (the column-chunk layout forms them once per
// chunk) and staged in LDS with their exponentials, 1024 tokens at a time
// with the running maximum rescaling the partial sums.  Chunks of VR
// vectors per row and TG token groups: NT = VR * TG threads, a multiple of
// 64 (pool_row_groups).
constexpr int kRowTile = 1024;
// Whole-row pooling needs at least this many (block, batch element) pairs;
// fewer take the column-chunk layout, which deals each pair to several
// workgroups.
constexpr int64_t kPoolRowMinGroups = 192;

template <typename T>
__global__ __launch_bounds__(512) void pool_row_kernel(const T* __restrict__ H,
                                                       const float* __restrict__ sp, int np,
                                                       float* __restrict__ s_out,
                                                       float* __restrict__ S, T* __restrict__ St,
                                                       float* __restrict__ stats, int Tn, int D,
                                                       int L, int nb, int TG,
                                                       float* __restrict__ zero, int64_t nzero) {
  constexpr int VE = Vec16<T>::N;
  constexpr int U = 8;
  typedef typename Vec16<T>::type vec;
  clear_share(zero, nzero);
  extern __shared__ float pdyn[];  // racc [TG][D], then sc [kRowTile]
  __shared__ float red[8];
  const int tid = threadIdx.x, nt = blockDim.x, nw = nt >> 6;
  const int VR = D / VE;
  const int v = tid % VR, tg = tid / VR;
  const int i = blockIdx.x, b = blockIdx.y;
  const int bs = i * L, be = min(bs + L, Tn);
  float* racc = pdyn;
  float* sc = pdyn + TG * D;
  const T* hb = H + ((int64_t)b * Tn) * D + v * VE;
  float m = -INFINITY, l = 0.f, acc[VE];
#pragma unroll
  for (int e = 0; e < VE; ++e) acc[e] = 0.f;
  for (int t0 = bs; t0 < be; t0 += kRowTile) {
    const int n = min(kRowTile, be - t0);
    // the tile's scores (the output projection left np partial sums each)
    float mx = -INFINITY;
    for (int t = tid; t < n; t += nt) {
      const int64_t row = (int64_t)b * Tn + t0 + t;
      const float x = score_sum(sp + row * np, np);
      sc[t] = x;
      s_out[row] = x;
      mx = fmaxf(mx, x);
    }
    mx = wave_max(mx);
    if ((tid & 63) == 0) red[tid >> 6] = mx;
    __syncthreads();
    float mn = m;
    for (int w = 0; w < nw; ++w) mn = fmaxf(mn, red[w]);
    __syncthreads();
    float ls = 0.f;
    for (int t = tid; t < n; t += nt) {
      const float e = __expf(sc[t] - mn);
      sc[t] = e;
      ls += e;
    }
    ls = wave_sum(ls);
    if ((tid & 63) == 0) red[tid >> 6] = ls;
    __syncthreads();
    float lt = 0.f;
    for (int w = 0; w < nw; ++w) lt += red[w];
    const float f = __expf(m - mn);
    l = l * f + lt;
    m = mn;
#pragma unroll
    for (int e = 0; e < VE; ++e) acc[e] *= f;
    if (tg < TG) {
      for (int k0 = tg; k0 < n; k0 += U * TG) {
        vec h[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int k = k0 + u * TG;
          h[u] = k < n ? load16(hb + (int64_t)(t0 + k) * D) : vec{};
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int k = k0 + u * TG;
          const float w = k < n ? sc[k] : 0.f;
#pragma unroll
          for (int e = 0; e < VE; ++e) acc[e] += w * to_f32(h[u][e]);
        }
      }
    }
    __syncthreads();  // sc[] and red[] are rewritten by the next tile
  }
  if (tg < TG) {
#pragma unroll
    for (int e = 0; e < VE; ++e) racc[tg * D + v * VE + e] = acc[e];
  }
  __syncthreads();
  const float inv = 1.0f / l;
  const int64_t brow = (int64_t)(b * nb + i);
  for (int c = tid; c < D; c += nt) {
    float sum = 0.f;
    for (int k = 0; k < TG; ++k) sum += racc[k * D + c];
    S[brow * D + c] = sum * inv;
    St[brow * D + c] = from_f32<T>(sum * inv);
  }
  if (tid == 0) {
    stats[brow * 2] = m;
    stats[brow * 2 + 1] = l;
  }
}

// ------------------------------------------------------------------ memory projection + scan
// Each workgroup owns 32 columns of one sequence and walks its N_b blocks in
// row tiles of 16: a small matrix product gives the tile's 16 x 32 outputs
// (the four waves take alternate 32-deep k steps and meet in LDS), then 32
// threads carry the decayed recurrence of their column through the tile.
//   forward:  Q = S W_m (A = S in the compute type, B = W_m [D, D] read
//             through LDS), and with Z_i = g Z_{i-1} + 1 the recurrences
//             N_i = g N_{i-1} + S_i and NP_i = g NP_{i-1} + Q_i give
//             M = N / Z (float32 and compute type) and P = M W_m = NP / Z
//             (the normalised decayed sum is linear, so scanning the
//             projections equals projecting the scan);
//   backward: dM = dP W_m^T (A = dP, B(k, n) = W_m[n, k], read directly),
//             then, from the last block down,
//               Qs_i = dM_i / Z_i + g Qs_{i+1}      (= dS_i = dN_i)
//               E_i  = -dM_i . M_i / Z_i + g E_{i+1} (= dZ_i, per column)
//             and dg = sum_{i>=1} Qs_i N_{i-1} + E_i Z_{i-1} with
//             N_{i-1} = M_{i-1} Z_{i-1}.
// A chunk that follows earlier blocks starts from their state (N, Z, and
// NP = Pc Z); the state after the last block goes to c.Nout / c.Zout, the
// gradients of that state enter the reverse scans at the last block, and
// E of the first block goes to c.e0.
// Z_i = 1 + g + ... + g^i + g^(i+1) zin (0-based i), where zin is the
// normaliser of the blocks before the first one (0 for none), with
// lg2 = log2(g) (g > 0).  The power underflows to 0 for long sequences,
// where Z_i has converged to 1 / (1 - g).
__device__ __forceinline__ float zsum(int i, float gamma, float lg2, float zin) {
  if (gamma == 0.f) return 1.f;
  const float gi = exp2f(lg2 * (float)(i + 1));
  return (1.f - gi) / (1.f - gamma) + gi * zin;
}

constexpr int kMsCols = 32, kMsRows = 16, kMsWaves = 8, kMsGroup = 4;

// Forward: W_m columns c0 .. c0+31 for rows kc .. kc+kn-1 are staged in LDS
// (dynamic, kc chunks of at most 64 KB); the k steps of a row tile are
// dealt to the eight waves round-robin and each wave loads kMsGroup steps'
// fragments before multiplying them, so that the loads overlap.
template <typename T, bool FWD>
__global__ __launch_bounds__(kMsWaves * 64) void memscan_kernel(
    const T* __restrict__ A, const T* __restrict__ Alo, const T* __restrict__ Wm,
    const float* __restrict__ S,
    float* __restrict__ M, T* __restrict__ Mt, float* __restrict__ P, const float* __restrict__ Min,
    float* __restrict__ dS, float* __restrict__ dgamma, int nb, int D, float gamma, int kcr,
    Carry cr, int lda) {
  typedef typename Frag<T>::type F;
  extern __shared__ __attribute__((aligned(16))) unsigned char dyn[];
  T* Bs = reinterpret_cast<T*>(dyn);  // [kcr][kMsCols] (forward only)
  __shared__ float part[kMsWaves][kMsRows][kMsCols];
  __shared__ float red[kMsWaves];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int c0 = blockIdx.x * kMsCols, b = blockIdx.y;
  const int nt = (nb + kMsRows - 1) / kMsRows;
  const int col = c0 + tid;
  const bool scol = tid < kMsCols && col < D;
  float N = 0.f, NP = 0.f, Z = 0.f, Qs = 0.f, E = 0.f, dg = 0.f;
  // this thread's column: its decay and its incoming normaliser
  float gam = (scol && cr.gvec) ? cr.gvec[col] : gamma;
  float lg2 = gam > 0.f ? log2f(gam) : 0.f;
  float zin = !cr.Zin ? 0.f : (!cr.zcol ? cr.Zin[b] : (scol ? cr.Zin[(int64_t)b * D + col] : 0.f));
  if constexpr (FWD) {
    Z = zin;
    if (scol && cr.Nin) {
      N = cr.Nin[(int64_t)b * D + col];
      NP = cr.Pc[(int64_t)b * D + col] * zin;
    }
  }
  // the gradients of the state after the last block (backward)
  float dn_last = 0.f, dz_last = 0.f;
  if constexpr (!FWD) {
    if (scol && cr.dNout) dn_last = cr.dNout[(int64_t)b * D + col];
    if (cr.dZout) {
      if (cr.zcol) dz_last = scol ? cr.dZout[(int64_t)b * D + col] : 0.f;
      else if (col == 0) dz_last = cr.dZout[b];
    }
  }
  // Loaded values pass through an empty asm before the row scans, so that
  // the compiler waits for their loads there, once: a wait inside a row
  // would also wait for the stores of the rows before it (vector memory
  // operations complete in order).
  asm volatile("" : "+v"(N), "+v"(NP), "+v"(Z), "+v"(gam), "+v"(lg2), "+v"(zin));
  asm volatile("" : "+v"(dn_last), "+v"(dz_last));

  for (int q = 0; q < nt; ++q) {
    const int rt = FWD ? q : nt - 1 - q;
    const int i0 = rt * kMsRows;
    const int arow = i0 + lr;
    const int64_t arow_off = ((int64_t)b * nb + (arow < nb ? arow : 0)) * lda;
    const T* ap = A + arow_off;
    // The tile's rows of S (forward) or M (backward, with the row before the
    // tile), loaded ahead of the product so that their latency overlaps it
    // and the recurrence below waits on no load.
    float rv[kMsRows], rprev = 0.f;
    if (scol) {
      const float* src = FWD ? S : Min;
#pragma unroll
      for (int k = 0; k < kMsRows; ++k)
        rv[k] = i0 + k < nb ? src[((int64_t)b * nb + i0 + k) * D + col] : 0.f;
      if (!FWD && i0 >= 1) rprev = Min[((int64_t)b * nb + i0 - 1) * D + col];
    }
    f32x4 acc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
    for (int kc = 0; kc < D; kc += (FWD ? kcr : D)) {
      const int kn = FWD ? min(kcr, D - kc) : D;
      if constexpr (FWD) {
        __syncthreads();
        // all of a batch's loads are issued before its LDS stores
        constexpr int VE = Vec16<T>::N;
        constexpr int VPR = kMsCols / VE;  // 16-byte vectors per staged row
        constexpr int UB = 8;
        typedef typename Vec16<T>::type V16;
        for (int e0 = tid; e0 < kn * VPR; e0 += UB * blockDim.x) {
          V16 v[UB];
#pragma unroll
          for (int u = 0; u < UB; ++u) {
            const int e = e0 + u * blockDim.x;
            const int kr = e / VPR, cv = (e % VPR) * VE;
            v[u] = (e < kn * VPR && c0 + cv < D) ? load16(Wm + (int64_t)(kc + kr) * D + c0 + cv)
                                                 : V16{};
          }
#pragma unroll
          for (int u = 0; u < UB; ++u) {
            const int e = e0 + u * blockDim.x;
            if (e < kn * VPR) store16(Bs + (e / VPR) * kMsCols + (e % VPR) * VE, v[u]);
          }
        }
        __syncthreads();
      }
      const int nks = kn / 32;
      for (int g0 = wave; g0 < nks; g0 += kMsWaves * kMsGroup) {
        F af[kMsGroup], bfr[kMsGroup][2];
#pragma unroll
        for (int u = 0; u < kMsGroup; ++u) {
          const int ks = g0 + u * kMsWaves;
          const bool on = ks < nks;
          const int kl = ks * 32 + lg * 8;  // within the chunk
          af[u] = (on && arow < nb) ? load_frag(ap + kc + kl) : F{};
#pragma unroll
          for (int ntl = 0; ntl < 2; ++ntl) {
            const int n = c0 + ntl * 16 + lr;
            if constexpr (FWD) {
#pragma unroll
              for (int e = 0; e < 8; ++e)
                bfr[u][ntl][e] = on ? Bs[(kl + e) * kMsCols + ntl * 16 + lr] : from_f32<T>(0.f);
            } else {
              bfr[u][ntl] = (on && n < D) ? load_frag(Wm + (int64_t)n * D + kc + kl) : F{};
            }
          }
        }
#pragma unroll
        for (int u = 0; u < kMsGroup; ++u)
#pragma unroll
          for (int ntl = 0; ntl < 2; ++ntl) acc[ntl] = mma16(bfr[u][ntl], af[u], acc[ntl]);
        if constexpr (!FWD) {
          // the low part of a hi + lo operand pair, against the same W_m fragments
          if (Alo) {
#pragma unroll
            for (int u = 0; u < kMsGroup; ++u) {
              const int ks = g0 + u * kMsWaves;
              af[u] = (ks < nks && arow < nb) ? load_frag(Alo + arow_off + kc + ks * 32 + lg * 8)
                                              : F{};
            }
#pragma unroll
            for (int u = 0; u < kMsGroup; ++u)
#pragma unroll
              for (int ntl = 0; ntl < 2; ++ntl) acc[ntl] = mma16(bfr[u][ntl], af[u], acc[ntl]);
          }
        }
      }
    }
    // lane holds row i0 + lr, columns 16 ntl + 4 lg + r of this wave's sum
#pragma unroll
    for (int ntl = 0; ntl < 2; ++ntl)
#pragma unroll
      for (int r = 0; r < 4; ++r) part[wave][lr][ntl * 16 + lg * 4 + r] = acc[ntl][r];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kMsRows; ++k) asm volatile("" : "+v"(rv[k]));
    asm volatile("" : "+v"(rprev));
    if (scol) {
#pragma unroll
      for (int k = 0; k < kMsRows; ++k) {
        const int ii = FWD ? k : kMsRows - 1 - k;
        const int i = i0 + ii;
        if (i >= nb) continue;
        float g = 0.f;
#pragma unroll
        for (int w = 0; w < kMsWaves; ++w) g += part[w][ii][tid];
        const int64_t off = ((int64_t)b * nb + i) * D + col;
        if constexpr (FWD) {
          N = gam * N + rv[ii];
          NP = gam * NP + g;
          Z = gam * Z + 1.f;
          const float rz = 1.f / Z;
          const float m = N * rz;
          M[off] = m;
          Mt[off] = from_f32<T>(m);
          P[off] = NP * rz;
        } else {
          const float z = zsum(i, gam, lg2, zin);
          const float m = rv[ii];
          Qs = g / z + gam * Qs;
          E = -g * m / z + gam * E;
          if (i == nb - 1) {
            Qs += dn_last;
            E += dz_last;
          }
          dS[off] = Qs;
          if (i >= 1) {
            const float zp = zsum(i - 1, gam, lg2, zin);
            const float mp = ii >= 1 ? rv[ii - 1] : rprev;
            dg += Qs * (mp * zp) + E * zp;
          } else if (cr.e0) {
            cr.e0[(int64_t)b * D + col] = E;
          }
        }
      }
    }
    __syncthreads();  // part[] is rewritten by the next row tile
  }
  if constexpr (FWD) {
    // the state after the last block
    if (scol && cr.Nout) cr.Nout[(int64_t)b * D + col] = N;
    if (scol && cr.Zout) {
      if (cr.zcol) cr.Zout[(int64_t)b * D + col] = Z;
      else if (tid == 0 && blockIdx.x == 0) cr.Zout[b] = Z;
    }
  }
  if constexpr (!FWD) {
    // this workgroup's share of the decay gradient, as one partial
    // (dg_part_rows): per channel, row b, its columns; else one value at
    // row b * gridDim.x + blockIdx.x
    if (cr.gvec) {
      if (scol && dgamma) dgamma[(int64_t)b * D + col] = dg;
    } else {
      const float v = wave_sum(dg);
      if (lane == 0) red[wave] = v;
      __syncthreads();
      if (tid == 0 && dgamma) {
        float t = 0.f;
        for (int w = 0; w < kMsWaves; ++w) t += red[w];
        dgamma[(int64_t)b * gridDim.x + blockIdx.x] = t;
      }
    }
  }
}

// ------------------------------------------------------------------ long scans
// For many blocks the memory path runs as two pieces: the W_m products as
// ordinary split-K matrix products, and the decayed scans below
// (memscan_kernel walks all blocks of a sequence through one matrix-core
// pass per 16 blocks, which serialises a long sequence).
//
// A scan is one launch over (64 columns, sequence): the workgroup owns its
// columns of the whole sequence, so no other workgroup's result is ever
// waited for, and every input is read once.  It walks the sequence in
// super-chunks of 128 blocks: each of its 8 waves scans 16 consecutive
// blocks of the super-chunk from a zero state (one lane per column, 256
// bytes per row of float32), the waves' aggregates meet in LDS, and each
// wave adds to its blocks the state entering its first block, decayed:
// with x_i = g x_{i-1} + y_i, a value is its local one plus g^(distance)
// times the carry.  The state leaving the super-chunk (the same sum, formed
// by every wave in the same order) enters the next one.  The first
// super-chunk starts from the state of the earlier blocks (zero for a
// whole sequence).
constexpr int kScCols = 64, kScWaves = 8, kScRows = 16, kScSuper = kScWaves * kScRows;
// The reverse scan: 16 waves of 8 blocks (more loads in flight per
// workgroup; its registers allow it, the forward's stores do not).
constexpr int kSbWaves = 16, kSbRows = 8, kSbSuper = kSbWaves * kSbRows;
// Up to this many blocks per sequence the fused kernel runs; beyond it, the
// scans above plus split-K matrix products (each split at least kMemMinK deep).
constexpr int kMemFusedMaxBlocks = 32, kMemMinK = 256;

// g^K for K a power of two: the decay across one wave's K blocks.
template <int K>
__device__ __forceinline__ float pow2k(float g) {
  static_assert(K >= 1 && (K & (K - 1)) == 0, "power of two");
#pragma unroll
  for (int k = 1; k < K; k *= 2) g *= g;
  return g;
}

// Forward: M = N / Z with N_i = g N_{i-1} + S_i (float32 and compute type).
// With Qp (one decay for all channels) also the projected summaries
// Q = S W_m, given as nq split-K partial products (stride qstride, added in
// order): NP_i = g NP_{i-1} + Q_i and P = NP / Z = M W_m.
template <typename T>
__global__ __launch_bounds__(kScCols * kScWaves) void scan_fwd_kernel(
    const float* __restrict__ S, float* __restrict__ M, T* __restrict__ Mt, int nb, int D,
    float gamma, Carry cr, const float* __restrict__ Qp, int nq, int64_t qstride,
    float* __restrict__ P) {
  __shared__ float wn[kScWaves][kScCols], wp[kScWaves][kScCols];
  const int c = threadIdx.x % kScCols, w = threadIdx.x / kScCols;
  const int col = blockIdx.x * kScCols + c;
  const bool on = col < D;
  const int b = blockIdx.y;
  const float gam = (on && cr.gvec) ? cr.gvec[col] : gamma;  // this column's decay
  const float lg2 = gam > 0.f ? log2f(gam) : 0.f;
  const float gw = pow2k<kScRows>(gam);  // across one wave's blocks
  const float zin = !cr.Zin ? 0.f
                    : (!cr.zcol ? cr.Zin[b] : (on ? cr.Zin[(int64_t)b * D + col] : 0.f));
  // the state entering the current super-chunk
  float sn = on && cr.Nin ? cr.Nin[(int64_t)b * D + col] : 0.f;
  float sp = on && Qp && cr.Nin ? cr.Pc[(int64_t)b * D + col] * zin : 0.f;
  const int64_t cbase = (int64_t)b * nb * D + col;
  for (int s0 = 0; s0 < nb; s0 += kScSuper) {
    const int a = s0 + w * kScRows;  // this wave's first block
    const int64_t off0 = cbase + (int64_t)a * D;
    float v[kScRows], q[kScRows];
#pragma unroll
    for (int r = 0; r < kScRows; ++r) {
      v[r] = on && a + r < nb ? S[off0 + (int64_t)r * D] : 0.f;
      q[r] = 0.f;
    }
    // the partial products one slice at a time, every row's load in flight
    for (int z = 0; Qp && z < nq; ++z) {
      float t[kScRows];
#pragma unroll
      for (int r = 0; r < kScRows; ++r)
        t[r] = on && a + r < nb ? Qp[z * qstride + off0 + (int64_t)r * D] : 0.f;
#pragma unroll
      for (int r = 0; r < kScRows; ++r) q[r] += t[r];
    }
    float n = 0.f, np = 0.f;
#pragma unroll
    for (int r = 0; r < kScRows; ++r) {
      n = gam * n + v[r];
      np = gam * np + q[r];
      v[r] = n;
      q[r] = np;
    }
    wn[w][c] = n;
    wp[w][c] = np;
    __syncthreads();
    // the state entering this wave's first block: the super-chunk's, then
    // the waves before this one
    float cn = sn, cp = sp;
    for (int j = 0; j < w; ++j) {
      cn = gw * cn + wn[j][c];
      cp = gw * cp + wp[j][c];
    }
    float f = gam;
    float zz = zsum(a, gam, lg2, zin);  // the normaliser, then its recurrence
#pragma unroll
    for (int r = 0; r < kScRows; ++r) {
      const int i = a + r;
      const float rz = 1.f / zz;
      zz = gam * zz + 1.f;
      if (on && i < nb) {
        const float nn = v[r] + f * cn;
        const float m = nn * rz;
        const int64_t off = off0 + (int64_t)r * D;
        M[off] = m;
        Mt[off] = from_f32<T>(m);
        if (Qp) P[off] = (q[r] + f * cp) * rz;
        if (i == nb - 1 && cr.Nout) cr.Nout[(int64_t)b * D + col] = nn;
      }
      f *= gam;
    }
    // the state leaving the super-chunk (only read when another follows,
    // which is then a whole one): every wave forms it in the same order
    for (int j = 0; j < kScWaves; ++j) {
      sn = gw * sn + wn[j][c];
      sp = gw * sp + wp[j][c];
    }
    __syncthreads();  // wn / wp are rewritten by the next super-chunk
  }
  if (cr.Zout && w == 0) {
    if (cr.zcol) {
      if (on) cr.Zout[(int64_t)b * D + col] = zsum(nb - 1, gam, lg2, zin);
    } else if (blockIdx.x == 0 && c == 0) {
      cr.Zout[b] = zsum(nb - 1, gam, lg2, zin);
    }
  }
}

// Reverse scans of the memory backward from dM (nq split-K partial products,
// stride qstride, added in order) and M:
//   Qs_i = dM_i / Z_i + g Qs_{i+1} (= dS_i),  E_i = -dM_i . M_i / Z_i + g E_{i+1},
//   dg = sum_{i>=1} Qs_i M_{i-1} Z_{i-1} + E_i Z_{i-1}   (one partial per workgroup;
//   per column with one decay per channel).
// Super-chunks from the last to the first; within one, the state entering a
// wave's last block comes from the later waves.  The gradients of a chunk's
// final state enter at the last block; E of the first block goes to cr.e0.
template <typename T>
__global__ __launch_bounds__(kScCols * kSbWaves) void scan_bwd_kernel(
    const float* __restrict__ dM, int nq, int64_t qstride, const float* __restrict__ M,
    float* __restrict__ dS, float* __restrict__ dgamma, int nb, int D, float gamma, Carry cr) {
  __shared__ float wq[kSbWaves][kScCols], we[kSbWaves][kScCols];
  __shared__ float red[kSbWaves];
  const int c = threadIdx.x % kScCols, w = threadIdx.x / kScCols;
  const int col = blockIdx.x * kScCols + c;
  const bool on = col < D;
  const int b = blockIdx.y;
  const float gam = (on && cr.gvec) ? cr.gvec[col] : gamma;  // this column's decay
  const float lg2 = gam > 0.f ? log2f(gam) : 0.f;
  const float gw = pow2k<kSbRows>(gam);  // across one wave's blocks
  const float zin = !cr.Zin ? 0.f
                    : (!cr.zcol ? cr.Zin[b] : (on ? cr.Zin[(int64_t)b * D + col] : 0.f));
  const int64_t cbase = (int64_t)b * nb * D + col;
  float sq = 0.f, se = 0.f;  // the state entering the current super-chunk from later blocks
  float dg = 0.f;
  for (int s0 = ((nb - 1) / kSbSuper) * kSbSuper; s0 >= 0; s0 -= kSbSuper) {
    const int a = s0 + w * kSbRows;
    const int64_t off0 = cbase + (int64_t)a * D;
    float x[kSbRows], y[kSbRows];
#pragma unroll
    for (int r = 0; r < kSbRows; ++r) x[r] = 0.f;
    for (int z = 0; z < nq; z += 2) {  // two slices' loads in flight at a time
      float t[kSbRows], u[kSbRows];
      const bool two = z + 1 < nq;
#pragma unroll
      for (int r = 0; r < kSbRows; ++r) {
        t[r] = on && a + r < nb ? dM[z * qstride + off0 + (int64_t)r * D] : 0.f;
        u[r] = two && on && a + r < nb ? dM[(z + 1) * qstride + off0 + (int64_t)r * D] : 0.f;
      }
#pragma unroll
      for (int r = 0; r < kSbRows; ++r) {
        x[r] += t[r];
        x[r] += u[r];
      }
    }
    float mm[kSbRows];
#pragma unroll
    for (int r = 0; r < kSbRows; ++r) mm[r] = on && a + r < nb ? M[off0 + (int64_t)r * D] : 0.f;
    // the memory of the block before this wave's first (its decay term)
    const float mprev = on && a >= 1 && a < nb ? M[off0 - D] : 0.f;
    // the normalisers of this wave's blocks: the closed form once, then the
    // recurrence; and the one before its first block (its decay term)
    float zs[kSbRows];
    float zz = zsum(a, gam, lg2, zin);
    const float zprev = a >= 1 ? zsum(a - 1, gam, lg2, zin) : 0.f;
#pragma unroll
    for (int r = 0; r < kSbRows; ++r) {
      const int i = a + r;
      const bool ok = on && i < nb;
      zs[r] = zz;
      const float rz = 1.f / zz;
      zz = gam * zz + 1.f;
      const float dm = x[r];
      x[r] = dm * rz;
      y[r] = -dm * mm[r] * rz;
      if (ok && i == nb - 1) {
        if (cr.dNout) x[r] += cr.dNout[(int64_t)b * D + col];
        if (cr.dZout) {
          if (cr.zcol) y[r] += cr.dZout[(int64_t)b * D + col];
          else if (col == 0) y[r] += cr.dZout[b];
        }
      }
    }
    float qq = 0.f, e = 0.f;
#pragma unroll
    for (int r = kSbRows - 1; r >= 0; --r) {
      qq = x[r] + gam * qq;
      e = y[r] + gam * e;
      x[r] = qq;
      y[r] = e;
    }
    wq[w][c] = qq;
    we[w][c] = e;
    __syncthreads();
    // the state entering this wave's last block: the super-chunk's, then
    // the later waves of this super-chunk
    float iq = sq, ie = se;
    for (int j = kSbWaves - 1; j > w; --j) {
      iq = wq[j][c] + gw * iq;
      ie = we[j][c] + gw * ie;
    }
    float f = gam;
#pragma unroll
    for (int r = kSbRows - 1; r >= 0; --r) {
      const int i = a + r;
      const float qs = x[r] + f * iq, es = y[r] + f * ie;
      f *= gam;
      if (on && i < nb) {
        dS[off0 + (int64_t)r * D] = qs;
        if (i >= 1) {
          const float zp = r > 0 ? zs[r > 0 ? r - 1 : 0] : zprev;
          const float mp = r > 0 ? mm[r > 0 ? r - 1 : 0] : mprev;
          dg += qs * (mp * zp) + es * zp;
        } else if (cr.e0) {
          cr.e0[(int64_t)b * D + col] = es;
        }
      }
    }
    // the state entering the previous super-chunk, the same in every wave
    for (int j = kSbWaves - 1; j >= 0; --j) {
      sq = wq[j][c] + gw * sq;
      se = we[j][c] + gw * se;
    }
    __syncthreads();  // wq / we are rewritten by the next super-chunk
  }
  // the decay gradient as partials (dg_part_rows): per channel, row b, this
  // workgroup's columns; else one value per workgroup
  if (cr.gvec) {  // the column's waves meet in LDS, in a fixed order
    wq[w][c] = dg;
    __syncthreads();
    if (w == 0 && on && dgamma) {
      float t = 0.f;
      for (int j = 0; j < kSbWaves; ++j) t += wq[j][c];
      dgamma[(int64_t)b * D + col] = t;
    }
    return;
  }
  const float v = wave_sum(dg);
  if (c == 0) red[w] = v;
  __syncthreads();
  if (threadIdx.x == 0 && dgamma) {
    float t = 0.f;
    for (int j = 0; j < kSbWaves; ++j) t += red[j];
    dgamma[(int64_t)b * gridDim.x + blockIdx.x] = t;
  }
}

// ------------------------------------------------------------------ look-back scans
// The long path's scans for few sequences (fewer than kLbMaxPairs sequence x
// 64-column slices, which the scans above would give one workgroup each):
// each sequence is cut into segments of kLbSeg blocks and every (segment,
// sequence, column slice) gets a workgroup, so the launch fills the chip.
// A workgroup scans its segment from a zero state, publishes the segment's
// aggregate (the state at its last block; the reverse scan's, at its first)
// for each of its columns, and reads the aggregates of the segments before
// it (after it, in reverse), which it folds in a fixed order (Horner over
// the segments, factor g^kLbSeg) into the state entering its segment; then
// it finishes its outputs as the scans above do with a super-chunk's carry.
// Reading every earlier aggregate (at most kLbMaxSeg - 1) rather than a
// running prefix keeps the result independent of timing: the same on every
// run.  Published words are 64 bits, the value's bits with a status word of
// 1 above them, written and read with device-scope atomics so that a
// workgroup on another XCD sees them; the launcher clears the words first.
// Workgroups are numbered segment first (the reverse scan from the last
// segment), so every segment a workgroup waits for belongs to a workgroup
// launched before it, which publishes before it waits itself; and the grid
// is kept to kLbMaxGroups small workgroups (256 threads, about 50
// registers, 2.5 KB of LDS), four per CU, which the chip holds at once.  A
// wait that exceeds kLbSpin polls gives up with NaN instead of hanging.  The
// records are cleared by the kernel before the scan on the same stream
// (pooling for the forward, the gate backward for the backward).
// Scalar decay and whole sequences only (no carried state).
constexpr int kLbWaves = 4, kLbRows = 4, kLbSeg = kLbWaves * kLbRows;
constexpr int kLbMaxPairs = 128, kLbMinSeg = 4, kLbMaxSeg = 64, kLbMaxGroups = 1024;
constexpr int kLbSpin = 1 << 18;

// Words of one segment's record: [quantity 0 | quantity 1] x 64 columns.
constexpr int kLbRec = 2 * kScCols;

__device__ __forceinline__ void lb_publish(uint64_t* p, float v) {
  const uint64_t w = (1ull << 32) | (uint64_t)__builtin_bit_cast(uint32_t, v);
  __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t lb_load(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// The value of a published word, polling until it is published.
__device__ __forceinline__ float lb_value(const uint64_t* p, uint64_t w) {
  for (int n = 0; (w >> 32) == 0; ++n) {
    if (n >= kLbSpin) return __builtin_nanf("");
    __builtin_amdgcn_s_sleep(2);
    w = lb_load(p);
  }
  return __builtin_bit_cast(float, (uint32_t)w);
}
// Fold of the published aggregates of segments j = j0, j0 + dj, ... (cnt of
// them) for one column and quantity: e = g * e + A_j in that order, sixteen
// loads in flight at a time.
__device__ __forceinline__ float lb_fold(const uint64_t* rec0, int j0, int dj, int cnt, float g) {
  float e = 0.f;
  for (int u0 = 0; u0 < cnt; u0 += 16) {
    uint64_t w[16];
#pragma unroll
    for (int u = 0; u < 16; ++u)
      w[u] = u0 + u < cnt ? lb_load(rec0 + (int64_t)(j0 + (u0 + u) * dj) * kLbRec) : 0ull;
#pragma unroll
    for (int u = 0; u < 16; ++u)
      if (u0 + u < cnt)
        e = fmaf(g, e, lb_value(rec0 + (int64_t)(j0 + (u0 + u) * dj) * kLbRec, w[u]));
  }
  return e;
}

// Forward (as scan_fwd_kernel without carried state): M = N / Z, and with Qp
// the projected summaries' scan P = NP / Z.  flags: B * ncs * nseg records,
// zero at launch.
template <typename T>
__global__ __launch_bounds__(kScCols * kLbWaves) void scan_fwd_lb_kernel(
    const float* __restrict__ S, float* __restrict__ M, T* __restrict__ Mt, int B, int nb, int D,
    float gamma, const float* __restrict__ Qp, int nq, int64_t qstride, float* __restrict__ P,
    uint64_t* __restrict__ flags, int nseg) {
  __shared__ float wn[kLbWaves][kScCols], wp[kLbWaves][kScCols], en[2][kScCols];
  const int c = threadIdx.x % kScCols, w = threadIdx.x / kScCols;
  const int ncs = (D + kScCols - 1) / kScCols;
  const int id = blockIdx.x;
  const int k = id / (B * ncs), b = (id / ncs) % B, x = id % ncs;
  const int col = x * kScCols + c;
  const bool on = col < D;
  const float lg2 = gamma > 0.f ? log2f(gamma) : 0.f;
  const float gw = pow2k<kLbRows>(gamma), gs = pow2k<kLbSeg>(gamma);
  const int a = k * kLbSeg + w * kLbRows;  // this wave's first block
  const int64_t off0 = (int64_t)b * nb * D + (int64_t)a * D + col;
  float v[kLbRows], q[kLbRows];
#pragma unroll
  for (int r = 0; r < kLbRows; ++r) {
    v[r] = on && a + r < nb ? S[off0 + (int64_t)r * D] : 0.f;
    q[r] = 0.f;
  }
  for (int z = 0; Qp && z < nq; ++z) {
#pragma unroll
    for (int r = 0; r < kLbRows; ++r)
      q[r] += on && a + r < nb ? Qp[z * qstride + off0 + (int64_t)r * D] : 0.f;
  }
  float n = 0.f, np = 0.f;
#pragma unroll
  for (int r = 0; r < kLbRows; ++r) {
    n = gamma * n + v[r];
    np = gamma * np + q[r];
    v[r] = n;
    q[r] = np;
  }
  wn[w][c] = n;
  wp[w][c] = np;
  __syncthreads();
  // wave 0: the aggregate of N, wave 1: of NP; publish it, then fold the
  // earlier segments' into the state entering this one
  uint64_t* rec0 = flags + ((int64_t)b * ncs + x) * nseg * kLbRec;
  if (w < (Qp ? 2 : 1)) {
    float agg = 0.f;
    for (int j = 0; j < kLbWaves; ++j) agg = gw * agg + (w == 0 ? wn[j][c] : wp[j][c]);
    if (k + 1 < nseg) lb_publish(rec0 + (int64_t)k * kLbRec + w * kScCols + c, agg);
    en[w][c] = k > 0 ? lb_fold(rec0 + w * kScCols + c, 0, 1, k, gs) : 0.f;
  }
  __syncthreads();
  float cn = en[0][c], cp = Qp ? en[1][c] : 0.f;
  for (int j = 0; j < w; ++j) {
    cn = gw * cn + wn[j][c];
    cp = gw * cp + wp[j][c];
  }
  float f = gamma;
  float zz = zsum(a, gamma, lg2, 0.f);
#pragma unroll
  for (int r = 0; r < kLbRows; ++r) {
    const int i = a + r;
    const float rz = 1.f / zz;
    zz = gamma * zz + 1.f;
    if (on && i < nb) {
      const float m = (v[r] + f * cn) * rz;
      const int64_t off = off0 + (int64_t)r * D;
      M[off] = m;
      Mt[off] = from_f32<T>(m);
      if (Qp) P[off] = (q[r] + f * cp) * rz;
    }
    f *= gamma;
  }
}

// Backward (as scan_bwd_kernel without carried state): dS from the nq
// partial slices of dM, and one decay-gradient partial per workgroup at
// dgamma[(b * ncs + x) * nseg + segment].  Segments are taken from the last.
template <typename T>
__global__ __launch_bounds__(kScCols * kLbWaves) void scan_bwd_lb_kernel(
    const float* __restrict__ dM, int nq, int64_t qstride, const float* __restrict__ M,
    float* __restrict__ dS, float* __restrict__ dgamma, int B, int nb, int D, float gamma,
    uint64_t* __restrict__ flags, int nseg) {
  __shared__ float wq[kLbWaves][kScCols], we[kLbWaves][kScCols], en[2][kScCols];
  __shared__ float red[kLbWaves];
  const int c = threadIdx.x % kScCols, w = threadIdx.x / kScCols;
  const int ncs = (D + kScCols - 1) / kScCols;
  const int id = blockIdx.x;
  const int k = nseg - 1 - id / (B * ncs), b = (id / ncs) % B, x = id % ncs;
  const int col = x * kScCols + c;
  const bool on = col < D;
  const float lg2 = gamma > 0.f ? log2f(gamma) : 0.f;
  const float gw = pow2k<kLbRows>(gamma), gs = pow2k<kLbSeg>(gamma);
  const int a = k * kLbSeg + w * kLbRows;
  const int64_t off0 = (int64_t)b * nb * D + (int64_t)a * D + col;
  float xr[kLbRows], yr[kLbRows], mm[kLbRows], zs[kLbRows];
#pragma unroll
  for (int r = 0; r < kLbRows; ++r) xr[r] = 0.f;
  for (int z = 0; z < nq; ++z) {
#pragma unroll
    for (int r = 0; r < kLbRows; ++r)
      xr[r] += on && a + r < nb ? dM[z * qstride + off0 + (int64_t)r * D] : 0.f;
  }
#pragma unroll
  for (int r = 0; r < kLbRows; ++r) mm[r] = on && a + r < nb ? M[off0 + (int64_t)r * D] : 0.f;
  const float mprev = on && a >= 1 && a < nb ? M[off0 - D] : 0.f;
  float zz = zsum(a, gamma, lg2, 0.f);
  const float zprev = a >= 1 ? zsum(a - 1, gamma, lg2, 0.f) : 0.f;
#pragma unroll
  for (int r = 0; r < kLbRows; ++r) {
    zs[r] = zz;
    const float rz = 1.f / zz;
    zz = gamma * zz + 1.f;
    const float dm = xr[r];
    xr[r] = dm * rz;
    yr[r] = -dm * mm[r] * rz;
  }
  float qq = 0.f, e = 0.f;
#pragma unroll
  for (int r = kLbRows - 1; r >= 0; --r) {
    qq = xr[r] + gamma * qq;
    e = yr[r] + gamma * e;
    xr[r] = qq;
    yr[r] = e;
  }
  wq[w][c] = qq;
  we[w][c] = e;
  __syncthreads();
  // wave 0: the aggregate of Qs, wave 1: of E (the state at the segment's
  // first block); publish it, then fold the later segments' (from the last)
  // into the state entering this segment's last block
  uint64_t* rec0 = flags + ((int64_t)b * ncs + x) * nseg * kLbRec;
  if (w < 2) {
    float agg = 0.f;
    for (int j = kLbWaves - 1; j >= 0; --j) agg = (w == 0 ? wq[j][c] : we[j][c]) + gw * agg;
    if (k > 0) lb_publish(rec0 + (int64_t)k * kLbRec + w * kScCols + c, agg);
    en[w][c] = k + 1 < nseg ? lb_fold(rec0 + w * kScCols + c, nseg - 1, -1, nseg - 1 - k, gs)
                            : 0.f;
  }
  __syncthreads();
  float iq = en[0][c], ie = en[1][c];
  for (int j = kLbWaves - 1; j > w; --j) {
    iq = wq[j][c] + gw * iq;
    ie = we[j][c] + gw * ie;
  }
  float f = gamma, dg = 0.f;
#pragma unroll
  for (int r = kLbRows - 1; r >= 0; --r) {
    const int i = a + r;
    const float qs = xr[r] + f * iq, es = yr[r] + f * ie;
    f *= gamma;
    if (on && i < nb) {
      dS[off0 + (int64_t)r * D] = qs;
      if (i >= 1) {
        const float zp = r > 0 ? zs[r > 0 ? r - 1 : 0] : zprev;
        const float mp = r > 0 ? mm[r > 0 ? r - 1 : 0] : mprev;
        dg += qs * (mp * zp) + es * zp;
      }
    }
  }
  const float vsum = wave_sum(dg);
  if (c == 0) red[w] = vsum;
  __syncthreads();
  if (threadIdx.x == 0 && dgamma) {
    float t = 0.f;
    for (int j = 0; j < kLbWaves; ++j) t += red[j];
    dgamma[((int64_t)b * ncs + x) * nseg + k] = t;
  }
}

// ------------------------------------------------------------------ gate backward
// dU = dY * Mc * G (1 - G) per element, and the block sum of dY * G, which is
// the gradient of the shifted memory, in the column-chunk layout.  The block
// sums are written already shifted back by one block (row i-1 holds block
// i's sum; the last row of each batch element is zero), in the compute type,
// as the left operand of the W_m backward products.  The first workgroup
// also clears zero_a / zero_b when given.  In a chunk that follows earlier blocks
// (Pc not null) block 0 was injected with Pc[b], and its sum goes to
// Pbar_c[b].
template <typename T>
__global__ __launch_bounds__(256) void gate_bwd_kernel(const T* __restrict__ dY,
                                                       const typename GateT<T>::type* __restrict__ G,
                                                       const float* __restrict__ P,
                                                       T* __restrict__ dU, T* __restrict__ Pbar,
                                                       float* __restrict__ zero_a, int na,
                                                       float* __restrict__ zero_b, int Tn, int D,
                                                       int L, int nb,
                                                       const float* __restrict__ Pc,
                                                       T* __restrict__ Pbar_c,
                                                       T* __restrict__ Pbar_lo,
                                                       T* __restrict__ Pbar_c_lo, int ldp) {
  constexpr int VE = Vec16<T>::N;
  typedef typename Vec16<T>::type vec;
  typedef typename GateT<T>::type GT;  // fp16 with bf16 activations
  typedef GT gvec __attribute__((ext_vector_type(VE)));
  __shared__ float racc[kTg][kVec * VE];
  clear_share(zero_a, na);
  if (blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0 && threadIdx.x == 0 && zero_b)
    *zero_b = 0.f;
  const int v = threadIdx.x % kVec, tg = threadIdx.x / kVec;
  const int i = blockIdx.x, b = blockIdx.y;
  const int c0 = blockIdx.z * kVec * VE;
  const int col = c0 + v * VE;
  const bool act = col < D;
  const int bs = i * L;
  const int be = min(bs + L, Tn);
  float c[VE], acc[VE];
#pragma unroll
  for (int e = 0; e < VE; ++e) {
    c[e] = 0.f;
    acc[e] = 0.f;
  }
  if (act && (i > 0 || Pc)) {
    const f32x4* pp = reinterpret_cast<const f32x4*>(
        i > 0 ? P + (int64_t)(b * nb + i - 1) * D + col : Pc + (int64_t)b * D + col);
#pragma unroll
    for (int q = 0; q < VE / 4; ++q) {
      const f32x4 w = pp[q];
#pragma unroll
      for (int r = 0; r < 4; ++r) c[q * 4 + r] = w[r];
    }
  }
  if (act) {
    constexpr int U = 2;
    for (int t0 = bs + tg; t0 < be; t0 += U * kTg) {
      vec dy[U];
      gvec g[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int t = t0 + u * kTg;
        const int64_t off = ((int64_t)b * Tn + t) * D + col;
        dy[u] = t < be ? load16(dY + off) : vec{};
        g[u] = t < be ? *reinterpret_cast<const gvec*>(G + off) : gvec{};
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int t = t0 + u * kTg;
        vec du;
#pragma unroll
        for (int e = 0; e < VE; ++e) {
          const float y = to_f32(dy[u][e]), gg = to_f32(g[u][e]);
          du[e] = from_f32<T>(y * c[e] * gg * (1.f - gg));
          acc[e] += y * gg;
        }
        if (t < be) store16(dU + ((int64_t)b * Tn + t) * D + col, du);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < VE; ++e) racc[tg][v * VE + e] = acc[e];
  __syncthreads();
  if (threadIdx.x < kVec * VE && c0 + (int)threadIdx.x < D) {
    const int cc = threadIdx.x;
    float sum = 0.f;
    for (int k = 0; k < kTg; ++k) sum += racc[k][cc];
    const int64_t dst = (int64_t)(b * nb + (i > 0 ? i - 1 : nb - 1)) * ldp + c0 + cc;
    // The sum as a pair hi + lo of the compute type (lo only for bf16): the
    // memory gradient takes both, the W_m weight gradient hi alone.
    const float v = i > 0 ? sum : 0.f;
    const T hi = from_f32<T>(v);
    Pbar[dst] = hi;
    if (Pbar_lo) Pbar_lo[dst] = from_f32<T>(v - to_f32(hi));
    if (i == 0 && Pbar_c) {
      const T hc = from_f32<T>(sum);
      Pbar_c[(int64_t)b * D + c0 + cc] = hc;
      if (Pbar_c_lo) Pbar_c_lo[(int64_t)b * D + c0 + cc] = from_f32<T>(sum - to_f32(hc));
    }
  }
}

// ------------------------------------------------------------------ chunk state
// One workgroup per sequence.  carry_prep: copy of the incoming state and its
// memory Nin / Zin in the compute type (the operand of the W_m product that
// feeds the chunk's first block); zero when there is no incoming state.  Z
// is one value per sequence, or one per channel (zcol).
template <typename T>
__global__ __launch_bounds__(256) void carry_prep_kernel(const float* __restrict__ Nu,
                                                         const float* __restrict__ Zu,
                                                         float* __restrict__ Nin,
                                                         float* __restrict__ Zin,
                                                         T* __restrict__ Mct,
                                                         float* __restrict__ Pc, int D, int zcol) {
  const int b = blockIdx.x;
  for (int c = threadIdx.x; c < D; c += blockDim.x) {
    const int64_t o = (int64_t)b * D + c;
    const float n = Nu ? Nu[o] : 0.f;
    const float z = Zu ? (zcol ? Zu[o] : Zu[b]) : 0.f;
    Nin[o] = n;
    if (zcol) Zin[o] = z;
    Mct[o] = from_f32<T>(z > 0.f ? n / z : 0.f);
    if (Pc) Pc[o] = 0.f;
  }
  if (!zcol && threadIdx.x == 0) Zin[b] = Zu ? Zu[b] : 0.f;
}

// carry_finish: gradients of the incoming state.  With M_in = Nin / Zin and
// dMc = dPc Wm^T its gradient through the first block's context,
//   N_0 = g Nin + S_0 and Z_0 = g Zin + 1 give
//   dNin = dMc / Zin + g dS_0,
//   dZin = sum_cols (g E_0 - dMc . M_in / Zin),
//   dgamma += sum_cols (dS_0 Nin + E_0 Zin)
// (the dMc terms vanish for an empty history, Zin = 0).
// With a per-channel decay (gvec) and normalisers (zcol) the same terms are
// kept per channel: dZin and the decay gradient are then [B, D] and [D].
__global__ __launch_bounds__(256) void carry_finish_kernel(
    const float* __restrict__ Nin, const float* __restrict__ Zin, const float* __restrict__ dMc,
    const float* __restrict__ dS, const float* __restrict__ e0, float* __restrict__ dNin,
    float* __restrict__ dZin, float* __restrict__ dgamma, int nb, int D, float gamma,
    const float* __restrict__ gvec, int zcol) {
  __shared__ float red[2][4];
  const int b = blockIdx.x, tid = threadIdx.x;
  float ez = 0.f, dg = 0.f;
  for (int c = tid; c < D; c += blockDim.x) {
    const int64_t o = (int64_t)b * D + c;
    const float z = zcol ? Zin[o] : Zin[b];
    const float gam = gvec ? gvec[c] : gamma;
    const float n = Nin[o], dm = dMc[o], e = e0[o];
    const float q = dS[(int64_t)b * nb * D + c];
    const float dmz = z > 0.f ? dm / z : 0.f;
    if (dNin) dNin[o] = dmz + gam * q;
    const float ezc = gam * e - (z > 0.f ? dmz * (n / z) : 0.f);
    const float dgc = q * n + e * z;
    if (zcol) {
      if (dZin) dZin[o] = ezc;
    } else {
      ez += ezc;
    }
    if (gvec) {
      if (dgamma) dgamma[o] = dgc;  // partial row b
    } else {
      dg += dgc;
    }
  }
  ez = wave_sum(ez);
  dg = wave_sum(dg);
  if ((tid & 63) == 0) {
    red[0][tid >> 6] = ez;
    red[1][tid >> 6] = dg;
  }
  __syncthreads();
  if (tid == 0) {
    const float tz = (red[0][0] + red[0][1]) + (red[0][2] + red[0][3]);
    const float tg = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
    if (dZin && !zcol) dZin[b] = tz;
    if (dgamma && !gvec) dgamma[b] = tg;  // partial row b
  }
}

// ------------------------------------------------------------------ pooling backward
// With a_t the block softmax weights and dS_i the summary gradient:
//   ds_t = a_t (dS_i . H[t] - dS_i . S_i),  dw_p = sum_t ds_t H[t].
// Each wave owns a segment of R consecutive rows of one block (the blocks'
// segments are numbered batch element, block, segment; a workgroup takes
// eight consecutive ones), so a launch has about B T / (8 R) workgroups
// whatever the block size, and a wave reads dS_i and S_i once for its R rows.
// The wave streams its rows TB at a time with the next TB rows' loads in
// flight while it forms the current rows' dot products with dS_i, writes a_t
// and ds_t (they feed the dH epilogue of the W_g backward product) and adds
// ds_t H[t] into registers.  The waves' sums meet in LDS in a fixed order and
// the workgroup's sum becomes one row of dwp_part; colsum_kernel adds the
// rows, so dw_p needs no atomics and comes out the same on every run.
// Rows a wave has in flight per load batch, by 16-byte vectors per lane and row.
constexpr int pool_tb(int nvj) { return nvj >= 4 ? 1 : 4 / nvj; }
template <int NVJ> struct PoolRows { static constexpr int TB = pool_tb(NVJ); };
constexpr int kPoolWaves = 8;

template <typename T, int NVJ>
__global__ __launch_bounds__(kPoolWaves * 64) void pool_bwd_kernel(
    const T* __restrict__ H, const float* __restrict__ s_in, const float* __restrict__ stats,
    const float* __restrict__ S, const float* __restrict__ dS, float* __restrict__ a_out,
    float* __restrict__ ds_out, float* __restrict__ dwp_part, int Bn, int Tn, int D, int L, int nb,
    int R, int nseg) {
  constexpr int VE = Vec16<T>::N;
  constexpr int TB = PoolRows<NVJ>::TB;
  constexpr int ROW = NVJ * 64 * VE;  // columns one wave covers
  typedef typename Vec16<T>::type vec;
  __shared__ float red[kPoolWaves / 2][ROW];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int Dv = D / VE;
  const int64_t seg = (int64_t)blockIdx.x * kPoolWaves + wave;
  const int64_t nall = (int64_t)Bn * nb * nseg;
  float pw[NVJ][VE];
#pragma unroll
  for (int j = 0; j < NVJ; ++j)
#pragma unroll
    for (int e = 0; e < VE; ++e) pw[j][e] = 0.f;

  if (seg < nall) {  // (uniform over the wave)
    const int b = (int)(seg / ((int64_t)nb * nseg));
    const int rem = (int)(seg - (int64_t)b * nb * nseg);
    const int i = rem / nseg, sg = rem % nseg;
    const int t0 = i * L + sg * R;
    const int t1 = min(min(t0 + R, i * L + L), Tn);
    const int64_t brow = (int64_t)(b * nb + i) * D;
    const T* hrow = H + (int64_t)b * Tn * D;

    float g[NVJ][VE];
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < NVJ; ++j) {
      const int v = lane + 64 * j;
      if (v < Dv) {
#pragma unroll
        for (int q = 0; q < VE / 4; ++q) {
          const f32x4 dv = *reinterpret_cast<const f32x4*>(dS + brow + v * VE + q * 4);
          const f32x4 sw = *reinterpret_cast<const f32x4*>(S + brow + v * VE + q * 4);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            g[j][q * 4 + r] = dv[r];
            ss += dv[r] * sw[r];
          }
        }
      } else {
#pragma unroll
        for (int e = 0; e < VE; ++e) g[j][e] = 0.f;
      }
    }
    const float mi = stats[(int64_t)(b * nb + i) * 2];
    const float li = stats[(int64_t)(b * nb + i) * 2 + 1];

    // rows t .. t+TB-1 (those below t1) into x and their scores into sv
    auto fetch = [&](vec(&x)[TB][NVJ], float(&sv)[TB], int t) {
#pragma unroll
      for (int k = 0; k < TB; ++k) {
        const bool tok = t + k < t1;
#pragma unroll
        for (int j = 0; j < NVJ; ++j) {
          const int v = lane + 64 * j;
          x[k][j] = tok && v < Dv ? load16(hrow + (int64_t)(t + k) * D + v * VE) : vec{};
        }
        sv[k] = tok ? s_in[(int64_t)b * Tn + t + k] : 0.f;
      }
    };
    float ssum = 0.f;  // wave_sum of ss, formed once the first rows are in flight
    auto consume = [&](vec(&x)[TB][NVJ], const float(&sv)[TB], int t) {
      float d[TB];
#pragma unroll
      for (int k = 0; k < TB; ++k) {
        float acc = 0.f;
#pragma unroll
        for (int j = 0; j < NVJ; ++j)
#pragma unroll
          for (int e = 0; e < VE; ++e) acc += g[j][e] * to_f32(x[k][j][e]);
        d[k] = wave_sum(acc);
      }
      // The rows stay packed until the second pass converts them again
      // (keeping both conversions would double the registers the rows take).
#pragma unroll
      for (int k = 0; k < TB; ++k)
#pragma unroll
        for (int j = 0; j < NVJ; ++j) asm volatile("" : "+v"(x[k][j]));
      float dsv = 0.f, av = 0.f;
#pragma unroll
      for (int k = 0; k < TB; ++k) {
        const bool tok = t + k < t1;
        const float a = __expf(sv[k] - mi) / li;
        const float ds = tok ? a * (d[k] - ssum) : 0.f;
        if (lane == k) {
          dsv = ds;
          av = a;
        }
#pragma unroll
        for (int j = 0; j < NVJ; ++j)
#pragma unroll
          for (int e = 0; e < VE; ++e) pw[j][e] += ds * to_f32(x[k][j][e]);
      }
      if (lane < TB && t + lane < t1) {
        const int64_t ti = (int64_t)b * Tn + t + lane;
        a_out[ti] = av;
        ds_out[ti] = dsv;
      }
    };
    vec xa[TB][NVJ], xb[TB][NVJ];
    float sa[TB], sb[TB];
    fetch(xa, sa, t0);
    ssum = wave_sum(ss);
    for (int t = t0; t < t1; t += 2 * TB) {
      if (t + TB < t1) fetch(xb, sb, t + TB);
      consume(xa, sa, t);
      if (t + TB >= t1) break;
      if (t + 2 * TB < t1) fetch(xa, sa, t + 2 * TB);
      consume(xb, sb, t + TB);
    }
  }
  if (!dwp_part) return;  // (uniform over the workgroup)

  // Pairwise tree over the waves: w += w + half, half = 4, 2, 1.
#pragma unroll
  for (int half = kPoolWaves / 2; half >= 1; half >>= 1) {
    if (wave >= half && wave < 2 * half) {
#pragma unroll
      for (int j = 0; j < NVJ; ++j)
#pragma unroll
        for (int e = 0; e < VE; ++e) red[wave - half][(lane + 64 * j) * VE + e] = pw[j][e];
    }
    __syncthreads();
    if (wave < half) {
#pragma unroll
      for (int j = 0; j < NVJ; ++j)
#pragma unroll
        for (int e = 0; e < VE; ++e) pw[j][e] += red[wave][(lane + 64 * j) * VE + e];
    }
    __syncthreads();
  }
  if (wave == 0) {
    float* row = dwp_part + (int64_t)blockIdx.x * D;
#pragma unroll
    for (int j = 0; j < NVJ; ++j) {
      const int v = lane + 64 * j;
      if (v < Dv) {
#pragma unroll
        for (int q = 0; q < VE / 4; ++q)
          *reinterpret_cast<f32x4*>(row + v * VE + q * 4) =
              f32x4{pw[j][q * 4], pw[j][q * 4 + 1], pw[j][q * 4 + 2], pw[j][q * 4 + 3]};
      }
    }
  }
}

// out[c] = sum over rows r < R of P[r][c] for 64 columns per workgroup and
// `per` rows per workgroup (blockIdx.y): thread (vector v, row group rg)
// adds rows rg, rg + 16, ... of its four columns, and the 16 row groups meet
// in LDS in a fixed order.  With more than one row range (gridDim.y > 1)
// each range writes its own row of `out` (stride N), which a second pass
// adds up.  One pass takes up to kColOnePass rows; longer inputs are first
// folded kColRows rows at a time.
constexpr int kColRows = 256;
constexpr int kColOnePass = 1024;
__global__ __launch_bounds__(256) void colsum_kernel(const float* __restrict__ P, int64_t R, int N,
                                                     int64_t per, float* __restrict__ out,
                                                     int accumulate) {
  __shared__ f32x4 red[16][16];
  const int v = threadIdx.x & 15, rg = threadIdx.x >> 4;
  const int c = blockIdx.x * 64 + v * 4;
  const int64_t r0 = (int64_t)blockIdx.y * per;
  const int64_t r1 = r0 + per < R ? r0 + per : R;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  if (c < N) {
    int64_t r = r0 + rg;
    for (; r + 48 < r1; r += 64) {
      const f32x4 a0 = *reinterpret_cast<const f32x4*>(P + r * N + c);
      const f32x4 a1 = *reinterpret_cast<const f32x4*>(P + (r + 16) * N + c);
      const f32x4 a2 = *reinterpret_cast<const f32x4*>(P + (r + 32) * N + c);
      const f32x4 a3 = *reinterpret_cast<const f32x4*>(P + (r + 48) * N + c);
      acc += (a0 + a1) + (a2 + a3);
    }
    for (; r < r1; r += 16) acc += *reinterpret_cast<const f32x4*>(P + r * N + c);
  }
  red[rg][v] = acc;
  __syncthreads();
  if (rg == 0 && c < N) {
    f32x4 sum = red[0][v];
    for (int k = 1; k < 16; ++k) sum += red[k][v];
    f32x4* dst = reinterpret_cast<f32x4*>(out + (int64_t)blockIdx.y * N + c);
    if (accumulate) sum += *dst;
    *dst = sum;
  }
}

// The decay gradient from its partials part[rows][Dp] (Dp = 1, or D with
// one decay per channel): out[c] (+)= sum over rows, in a fixed order.
// Dp = 1: one workgroup; thread t adds rows t, t + 256, ... in order, then
// the waves' sums and the four wave results in a fixed order.  Dp > 1:
// workgroup = 64 columns, wave w adds rows w, w + 4, ... in order, the four
// sums meet in LDS.
__global__ __launch_bounds__(256) void dgamma_reduce_kernel(const float* __restrict__ part,
                                                            int rows, int Dp,
                                                            float* __restrict__ out,
                                                            int accumulate) {
  __shared__ float red[4][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (Dp == 1) {
    float t = 0.f;
#pragma unroll 8
    for (int r = threadIdx.x; r < rows; r += 256) t += part[r];
    t = wave_sum(t);
    if (lane == 0) red[wave][0] = t;
    __syncthreads();
    if (threadIdx.x == 0) {
      const float v = (red[0][0] + red[1][0]) + (red[2][0] + red[3][0]);
      out[0] = accumulate ? out[0] + v : v;
    }
    return;
  }
  const int c = blockIdx.x * 64 + lane;
  float t = 0.f;
  if (c < Dp)
    for (int r = wave; r < rows; r += 4) t += part[(int64_t)r * Dp + c];
  red[wave][lane] = t;
  __syncthreads();
  if (wave == 0 && c < Dp) {
    const float v = (red[0][lane] + red[1][lane]) + (red[2][lane] + red[3][lane]);
    out[c] = accumulate ? out[c] + v : v;
  }
}

__global__ void zero_two_kernel(float* a, int64_t na, float* b, int64_t nb) {
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < na + nb;
       k += (int64_t)gridDim.x * blockDim.x) {
    if (k < na) {
      if (a) a[k] = 0.f;
    } else if (b) {
      b[k - na] = 0.f;
    }
  }
}

__global__ void fill_kernel(float* p, int64_t n, float v) {
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < n;
       k += (int64_t)gridDim.x * blockDim.x)
    p[k] = v;
}

int nvj_for(int Dv) {
  const int n = (Dv + 63) / 64;
  return n <= 1 ? 1 : n <= 2 ? 2 : n <= 4 ? 4 : 8;
}

template <typename E>
hipError_t pool_fwd_t(const void* H, const float* sp, int np, float* s_out, float* S, void* St,
                      float* stats, int B, int T, int D, int L, float* zero, int64_t nzero,
                      hipStream_t s) {
  const int nb = (T + L - 1) / L;
  if ((int64_t)B * nb >= kPoolRowMinGroups) {
    // whole rows: VR vectors per row, TG token groups, VR * TG threads a
    // multiple of 64 and at least 256 (or VR itself when larger)
    const int VR = D / Vec16<E>::N;
    int TG = VR >= 256 ? 1 : (256 + VR - 1) / VR;
    while ((VR * TG) % 64) ++TG;
    const size_t lds = ((size_t)TG * D + kRowTile) * sizeof(float);
    hipLaunchKernelGGL(pool_row_kernel<E>, dim3(nb, B), dim3(VR * TG), lds, s, (const E*)H, sp, np,
                       s_out, S, (E*)St, stats, T, D, L, nb, TG, zero, nzero);
    return hipGetLastError();
  }
  const int cw = kVec * Vec16<E>::N;
  hipLaunchKernelGGL(pool_fwd_kernel<E>, dim3(nb, B, (D + cw - 1) / cw), dim3(kVec * kTg), 0, s,
                     (const E*)H, sp, np, s_out, S, (E*)St, stats, T, D, L, nb, zero, nzero);
  return hipGetLastError();
}

// Rows per wave (R), segments per block and workgroups of the pooling
// backward: R is a multiple of the rows a wave has in flight, chosen for
// about 1024 workgroups, but at least 8 rows (at most 64, at most a block).
// Short inputs thus leave CUs free for the weight-gradient products that run
// beside this kernel on the second stream: at B = 8, T = 1024, D = 768, 512
// workgroups of 2 rows per wave made this kernel 0.8 us faster and the step
// 9.5 us slower than 128 workgroups.
struct PoolBwdShape {
  int R, nseg;
  int64_t nwg;
};
template <typename E>
PoolBwdShape pool_bwd_shape(int B, int D, int L, int T) {
  const int tb = pool_tb(nvj_for(D / Vec16<E>::N));
  const int nb = (T + L - 1) / L;
  const int lb = L < T ? L : T;
  const int64_t want = (int64_t)B * T / (kPoolWaves * 1024);
  int64_t r = (want + tb - 1) / tb * tb;
  r = r < 8 ? 8 : r > 64 ? 64 : r;
  const int64_t lr = (lb + tb - 1) / tb * tb;
  if (r > lr) r = lr;
  PoolBwdShape p;
  p.R = (int)r;
  p.nseg = (lb + p.R - 1) / p.R;
  p.nwg = ((int64_t)B * nb * p.nseg + kPoolWaves - 1) / kPoolWaves;
  return p;
}

template <typename E, int NV>
hipError_t pool_bwd_nv(const void* H, const float* s_in, const float* stats, const float* S,
                       const float* dS, float* a_out, float* ds_out, float* dwp_part, int B,
                       int T, int D, int L, hipStream_t s) {
  const int nb = (T + L - 1) / L;
  const PoolBwdShape p = pool_bwd_shape<E>(B, D, L, T);
  if (p.nwg > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((pool_bwd_kernel<E, NV>), dim3((unsigned)p.nwg), dim3(kPoolWaves * 64), 0,
                     s, (const E*)H, s_in, stats, S, dS, a_out, ds_out, dwp_part, B, T, D, L, nb,
                     p.R, p.nseg);
  return hipGetLastError();
}

template <typename E>
hipError_t pool_bwd_t(const void* H, const float* s_in, const float* stats, const float* S,
                      const float* dS, float* a_out, float* ds_out, float* dwp_part, int B, int T,
                      int D, int L, hipStream_t s) {
  switch (nvj_for(D / Vec16<E>::N)) {
    case 1: return pool_bwd_nv<E, 1>(H, s_in, stats, S, dS, a_out, ds_out, dwp_part, B, T, D, L, s);
    case 2: return pool_bwd_nv<E, 2>(H, s_in, stats, S, dS, a_out, ds_out, dwp_part, B, T, D, L, s);
    case 4: return pool_bwd_nv<E, 4>(H, s_in, stats, S, dS, a_out, ds_out, dwp_part, B, T, D, L, s);
    default: return pool_bwd_nv<E, 8>(H, s_in, stats, S, dS, a_out, ds_out, dwp_part, B, T, D, L, s);
  }
}

template <typename E>
hipError_t gate_bwd_t(const void* dY, const void* G, const float* P, void* dU, void* Pbar,
                      void* Pbar_lo, float* zero_a, int na, float* zero_b, int B, int T, int D,
                      int L, const float* Pc, void* Pbar_c, void* Pbar_c_lo, hipStream_t s) {
  const int nb = (T + L - 1) / L;
  const int cw = kVec * Vec16<E>::N;
  hipLaunchKernelGGL(gate_bwd_kernel<E>, dim3(nb, B, (D + cw - 1) / cw), dim3(kVec * kTg), 0, s,
                     (const E*)dY, (const typename GateT<E>::type*)G, P, (E*)dU, (E*)Pbar, zero_a,
                     na, zero_b, T, D, L,
                     nb, Pc, (E*)Pbar_c, Pbar_lo ? (E*)Pbar + D : (E*)nullptr, (E*)Pbar_c_lo,
                     Pbar_lo ? 2 * D : D);
  return hipGetLastError();
}

}  // namespace

hipError_t pool_fwd(DType dt, const void* H, const float* sp, int np, float* s_out, float* S,
                    void* St, float* stats, int B, int T, int D, int L, float* zero,
                    int64_t nzero, hipStream_t s) {
  if (dt == DType::BF16)
    return pool_fwd_t<bf16>(H, sp, np, s_out, S, St, stats, B, T, D, L, zero, nzero, s);
  return pool_fwd_t<float>(H, sp, np, s_out, S, St, stats, B, T, D, L, zero, nzero, s);
}

bool mem_fused(int nb, bool per_channel) { return nb <= kMemFusedMaxBlocks && !per_channel; }

// The long path's W_m products keep their split-K partial products (one
// slice per split, a single slice when there is one split) for the scans,
// which add them in a fixed order: the forward's Q = St W_m, and the
// backward's dM = [Pbar | Pbar_lo] [Wm^T; Wm^T] (one product over 2D).
// Bytes of the W_m products' split-K slices.
size_t mem_slice_bytes(int B, int nb, int D) {
  const int sp = std::max(gemm_splitk_splits(B * nb, D, D, kMemMinK),
                          gemm_splitk_splits(B * nb, D, 2 * D, kMemMinK));
  return ((size_t)sp * B * nb * D * sizeof(float) + 255) / 256 * 256;
}

bool has_carry(const Carry& c) {
  return c.Nin || c.Zin || c.Pc || c.Nout || c.Zout || c.dNout || c.dZout || c.e0;
}

// Segments of the look-back scans, or 0 where the scans above serve.
int lb_nseg(int B, int nb, int D, bool per_channel, bool carry) {
  if (per_channel || carry || mem_fused(nb, per_channel)) return 0;
  const int ncs = (D + kScCols - 1) / kScCols;
  if ((int64_t)B * ncs >= kLbMaxPairs) return 0;
  const int ns = (nb + kLbSeg - 1) / kLbSeg;
  if ((int64_t)B * ncs * ns > kLbMaxGroups) return 0;
  return ns >= kLbMinSeg && ns <= kLbMaxSeg ? ns : 0;
}

// Words of the look-back records.
int64_t lb_words(int B, int D, int nseg) {
  return (int64_t)B * ((D + kScCols - 1) / kScCols) * nseg * kLbRec;
}

float* mem_lb_flags(float* part, int B, int nb, int D, bool per_channel, bool carry,
                    int64_t* nfloat) {
  const int ns = lb_nseg(B, nb, D, per_channel, carry);
  *nfloat = ns ? 2 * lb_words(B, D, ns) : 0;
  return ns ? reinterpret_cast<float*>(reinterpret_cast<char*>(part) + mem_slice_bytes(B, nb, D))
            : nullptr;
}

size_t mem_part_bytes(int B, int nb, int D, bool per_channel) {
  if (mem_fused(nb, per_channel)) return 0;
  const int ns = lb_nseg(B, nb, D, per_channel, false);
  return mem_slice_bytes(B, nb, D) + (ns ? (size_t)lb_words(B, D, ns) * 8 : 0);
}

// One scan launch over grid (columns / 64, B), or the look-back scan over
// every (segment, sequence, column slice) for few sequences, whose records
// (after the split-K slices in `part`, mem_lb_flags) an earlier kernel on
// the stream has cleared.
template <typename T>
hipError_t scan_fwd_run(const float* S, float* M, T* Mt, int B, int nb, int D, float gamma,
                        const Carry& c, const float* Qp, int nq, float* P, float* part,
                        hipStream_t s) {
  const int ns = lb_nseg(B, nb, D, c.gvec != nullptr, has_carry(c));
  if (ns) {
    uint64_t* fl = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(part) +
                                                mem_slice_bytes(B, nb, D));
    const int nwg = B * ((D + kScCols - 1) / kScCols) * ns;
    hipLaunchKernelGGL(scan_fwd_lb_kernel<T>, dim3(nwg), dim3(kScCols * kLbWaves), 0, s, S, M,
                       Mt, B, nb, D, gamma, Qp, nq, (int64_t)B * nb * D, P, fl, ns);
    return hipGetLastError();
  }
  const dim3 grid((D + kScCols - 1) / kScCols, B);
  hipLaunchKernelGGL(scan_fwd_kernel<T>, grid, dim3(kScCols * kScWaves), 0, s, S, M, Mt, nb, D,
                     gamma, c, Qp, nq, (int64_t)B * nb * D, P);
  return hipGetLastError();
}

template <typename T>
hipError_t scan_bwd_run(const float* dM, int nq, const float* M, float* dS, float* dgamma, int B,
                        int nb, int D, float gamma, const Carry& c, float* part, hipStream_t s) {
  const int ns = lb_nseg(B, nb, D, c.gvec != nullptr, has_carry(c));
  if (ns) {
    uint64_t* fl = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(part) +
                                                mem_slice_bytes(B, nb, D));
    const int nwg = B * ((D + kScCols - 1) / kScCols) * ns;
    hipLaunchKernelGGL(scan_bwd_lb_kernel<T>, dim3(nwg), dim3(kScCols * kLbWaves), 0, s, dM, nq,
                       (int64_t)B * nb * D, M, dS, dgamma, B, nb, D, gamma, fl, ns);
    return hipGetLastError();
  }
  const dim3 grid((D + kScCols - 1) / kScCols, B);
  hipLaunchKernelGGL(scan_bwd_kernel<T>, grid, dim3(kScCols * kSbWaves), 0, s, dM, nq,
                     (int64_t)B * nb * D, M, dS, dgamma, nb, D, gamma, c);
  return hipGetLastError();
}

// The long path in its steps (mem_fused false), each one launch sequence:
// mem_fwd_proj the W_m product before the scans (one decay: Q = St W_m as
// split-K partials, *nq slices) or after them (one decay per channel:
// P = M W_m), mem_fwd_scan the two scan passes.
hipError_t mem_fwd_proj(DType dt, const void* St, const void* Wm, const void* Mt, float* P,
                        float* part, int B, int nb, int D, bool per_channel, int* nq,
                        hipStream_t s) {
  *nq = 0;
  if (!per_channel) {
    GemmDesc g{B * nb, D, D, St, D, false, {Wm, nullptr, nullptr}, D, true, kSegNone, 0, 1};
    return gemm_splitk_product(dt, g, part, part, nullptr, nullptr, D, D, false, kMemMinK, nq, s);
  }
  GemmDesc g{B * nb, D, D, Mt, D, false, {Wm, nullptr, nullptr}, D, true, kSegNone, 0, 1};
  return gemm_splitk(dt, g, part, P, nullptr, nullptr, D, D, false, kMemMinK, s);
}

hipError_t mem_fwd_scan(DType dt, const float* S, float* M, void* Mt, float* P, float* part, int nq,
                        int B, int nb, int D, float gamma, const Carry& c, hipStream_t s) {
  const float* Qp = c.gvec ? nullptr : part;
  float* Pout = c.gvec ? nullptr : P;
  if (dt == DType::BF16)
    return scan_fwd_run<bf16>(S, M, (bf16*)Mt, B, nb, D, gamma, c, Qp, c.gvec ? 0 : nq, Pout,
                              part, s);
  return scan_fwd_run<float>(S, M, (float*)Mt, B, nb, D, gamma, c, Qp, c.gvec ? 0 : nq, Pout,
                             part, s);
}

hipError_t mem_fwd(DType dt, const void* St, const void* Wm, const float* S, float* M, void* Mt,
                   float* P, float* part, int B, int nb, int D, float gamma, const Carry& c,
                   hipStream_t s) {
  if (!mem_fused(nb, c.gvec != nullptr)) {
    // One decay: Q = St W_m, then one scan of S and Q gives M and P = M W_m
    // (the decayed sum is linear).  One decay per channel: W_m mixes
    // channels, so the scan of S comes first and P = M W_m is a product.
    int nq = 0;
    const bool pc = c.gvec != nullptr;
    hipError_t e = hipSuccess;
    if (!pc) e = mem_fwd_proj(dt, St, Wm, Mt, P, part, B, nb, D, false, &nq, s);
    if (e == hipSuccess) e = mem_fwd_scan(dt, S, M, Mt, P, part, nq, B, nb, D, gamma, c, s);
    if (e == hipSuccess && pc) e = mem_fwd_proj(dt, St, Wm, Mt, P, part, B, nb, D, true, &nq, s);
    return e;
  }
  dim3 grid((D + kMsCols - 1) / kMsCols, B);
  const int es = dt == DType::BF16 ? 2 : 4;
  int kcr = (64 * 1024) / (kMsCols * es);  // staged W_m rows per chunk (64 KB)
  if (kcr > D) kcr = D;
  const size_t lds = (size_t)kcr * kMsCols * es;
  if (dt == DType::BF16)
    hipLaunchKernelGGL((memscan_kernel<bf16, true>), grid, dim3(kMsWaves * 64), lds, s,
                       (const bf16*)St, (const bf16*)nullptr, (const bf16*)Wm, S, M, (bf16*)Mt, P,
                       nullptr, nullptr, nullptr, nb, D, gamma, kcr, c, D);
  else
    hipLaunchKernelGGL((memscan_kernel<float, true>), grid, dim3(kMsWaves * 64), lds, s,
                       (const float*)St, (const float*)nullptr, (const float*)Wm, S, M,
                       (float*)Mt, P, nullptr, nullptr, nullptr, nb, D, gamma, kcr, c, D);
  return hipGetLastError();
}

hipError_t gate_bwd(DType dt, const void* dY, const void* G, const float* P, void* dU,
                    void* Pbar, void* Pbar_lo, float* zero_a, int na, float* zero_b, int B, int T,
                    int D, int L, const float* Pc, void* Pbar_c, void* Pbar_c_lo, hipStream_t s) {
  if (dt == DType::BF16)
    return gate_bwd_t<bf16>(dY, G, P, dU, Pbar, Pbar_lo, zero_a, na, zero_b, B, T, D, L, Pc,
                            Pbar_c, Pbar_c_lo, s);
  return gate_bwd_t<float>(dY, G, P, dU, Pbar, nullptr, zero_a, na, zero_b, B, T, D, L, Pc,
                           Pbar_c, nullptr, s);
}

// The long path's backward steps: mem_bwd_proj dM = dP W_m^T as split-K
// partials (dP = hi + lo: two products, their slices one after the other;
// *nq slices in all), mem_bwd_scan the reverse scans, which add them up.
hipError_t mem_bwd_proj(DType dt, const void* Pbar, const void* Pbar_lo, const void* Wm,
                        float* part, int B, int nb, int D, int* nq, hipStream_t s) {
  *nq = 0;
  if (dt == DType::BF16 && Pbar_lo) {
    // rows [hi | lo] (2D wide) against [W_m^T; W_m^T]: one product over
    // K = 2D whose B is the same matrix for both halves of K
    GemmDesc g{B * nb, D, 2 * D, Pbar, 2 * D, false, {Wm, Wm, nullptr}, D, false, kSegK, D, 1};
    return gemm_splitk_product(dt, g, part, part, nullptr, nullptr, D, D, false, kMemMinK, nq, s);
  }
  GemmDesc g{B * nb, D, D, Pbar, D, false, {Wm, nullptr, nullptr}, D, false, kSegNone, 0, 1};
  return gemm_splitk_product(dt, g, part, part, nullptr, nullptr, D, D, false, kMemMinK, nq, s);
}

hipError_t mem_bwd_scan(DType dt, const float* M, float* dS, float* dgpart, float* part, int nq,
                        int B, int nb, int D, float gamma, const Carry& c, hipStream_t s) {
  if (dt == DType::BF16)
    return scan_bwd_run<bf16>(part, nq, M, dS, dgpart, B, nb, D, gamma, c, part, s);
  return scan_bwd_run<float>(part, nq, M, dS, dgpart, B, nb, D, gamma, c, part, s);
}

hipError_t mem_bwd(DType dt, const void* Pbar, const void* Pbar_lo, const void* Wm,
                   const float* M, float* dS, float* dgpart, float* dM, float* part, int B, int nb,
                   int D, float gamma, const Carry& c, hipStream_t s) {
  if (dt != DType::BF16) Pbar_lo = nullptr;
  (void)dM;
  if (!mem_fused(nb, c.gvec != nullptr)) {
    int nq = 0;
    hipError_t e = mem_bwd_proj(dt, Pbar, Pbar_lo, Wm, part, B, nb, D, &nq, s);
    if (e != hipSuccess) return e;
    return mem_bwd_scan(dt, M, dS, dgpart, part, nq, B, nb, D, gamma, c, s);
  }
  dim3 grid((D + kMsCols - 1) / kMsCols, B);
  if (dt == DType::BF16)
    hipLaunchKernelGGL((memscan_kernel<bf16, false>), grid, dim3(kMsWaves * 64), 0, s,
                       (const bf16*)Pbar, Pbar_lo ? (const bf16*)Pbar + D : (const bf16*)nullptr,
                       (const bf16*)Wm, nullptr, nullptr, nullptr, nullptr, M, dS, dgpart, nb, D,
                       gamma, 0, c, Pbar_lo ? 2 * D : D);
  else
    hipLaunchKernelGGL((memscan_kernel<float, false>), grid, dim3(kMsWaves * 64), 0, s,
                       (const float*)Pbar, (const float*)nullptr, (const float*)Wm, nullptr,
                       nullptr, nullptr, nullptr, M, dS, dgpart, nb, D, gamma, 0, c, D);
  return hipGetLastError();
}

hipError_t carry_prep(DType dt, const float* Nu, const float* Zu, float* Nin, float* Zin,
                      void* Mct, float* Pc, int B, int D, bool zcol, hipStream_t s) {
  if (dt == DType::BF16)
    hipLaunchKernelGGL(carry_prep_kernel<bf16>, dim3(B), dim3(256), 0, s, Nu, Zu, Nin, Zin,
                       (bf16*)Mct, Pc, D, zcol ? 1 : 0);
  else
    hipLaunchKernelGGL(carry_prep_kernel<float>, dim3(B), dim3(256), 0, s, Nu, Zu, Nin, Zin,
                       (float*)Mct, Pc, D, zcol ? 1 : 0);
  return hipGetLastError();
}

size_t carry_part_bytes(int B, int D) { return gemm_splitk_partial_bytes(B, D, D, kMemMinK); }

hipError_t carry_proj(DType dt, const void* A, const void* Wm, float* out, float* part,
                      bool transposed, bool accumulate, int B, int D, hipStream_t s) {
  // B(k, n) = Wm[k, n] (Pc = Mct Wm) or Wm[n, k] (dMc = Pbar_c Wm^T).
  GemmDesc g{B, D, D, A, D, false, {Wm, nullptr, nullptr}, D, !transposed, kSegNone, 0, 1};
  return gemm_splitk(dt, g, part, out, nullptr, nullptr, D, D, accumulate, kMemMinK, s);
}

hipError_t carry_finish(const float* Nin, const float* Zin, const float* dMc, const float* dS,
                        const float* e0, float* dNin, float* dZin, float* dgamma, int B, int nb,
                        int D, float gamma, const float* gvec, bool zcol, hipStream_t s) {
  if (!dNin && !dZin && !dgamma) return hipSuccess;
  hipLaunchKernelGGL(carry_finish_kernel, dim3(B), dim3(256), 0, s, Nin, Zin, dMc, dS, e0, dNin,
                     dZin, dgamma, nb, D, gamma, gvec, zcol ? 1 : 0);
  return hipGetLastError();
}

hipError_t pool_bwd(DType dt, const void* H, const float* s_in, const float* stats,
                    const float* S, const float* dS, float* a_out, float* ds_out,
                    float* dwp_part, int B, int T, int D, int L, hipStream_t s) {
  if (dt == DType::BF16)
    return pool_bwd_t<bf16>(H, s_in, stats, S, dS, a_out, ds_out, dwp_part, B, T, D, L, s);
  return pool_bwd_t<float>(H, s_in, stats, S, dS, a_out, ds_out, dwp_part, B, T, D, L, s);
}

// Rows of dw_p partial sums the pooling backward writes (one per workgroup).
int64_t pool_rows(DType dt, int B, int T, int D, int L) {
  return dt == DType::BF16 ? pool_bwd_shape<bf16>(B, D, L, T).nwg
                           : pool_bwd_shape<float>(B, D, L, T).nwg;
}

int64_t pool_bwd_partial_rows(DType dt, int B, int T, int D, int L) {
  int64_t r = pool_rows(dt, B, T, D, L), all = r;
  while (r > kColOnePass) {  // the reduction's intermediate rows
    r = (r + kColRows - 1) / kColRows;
    all += r;
  }
  return all;
}

hipError_t pool_dwp(float* dwp_part, DType dt, int B, int T, int D, int L, float* dwp,
                    bool accumulate, hipStream_t s) {
  if (!dwp) return hipSuccess;
  int64_t R = pool_rows(dt, B, T, D, L);
  float* in = dwp_part;
  // Each pass folds kColRows rows into one, in a fixed order, until one
  // pass can take the rest.
  while (R > kColOnePass) {
    const int64_t ranges = (R + kColRows - 1) / kColRows;
    if (ranges > 65535) return hipErrorInvalidValue;
    float* out = in + R * D;
    hipLaunchKernelGGL(colsum_kernel, dim3((D + 63) / 64, (unsigned)ranges), dim3(256), 0, s,
                       (const float*)in, R, D, (int64_t)kColRows, out, 0);
    in = out;
    R = ranges;
  }
  hipLaunchKernelGGL(colsum_kernel, dim3((D + 63) / 64, 1), dim3(256), 0, s, (const float*)in, R,
                     D, R, dwp, accumulate ? 1 : 0);
  return hipGetLastError();
}

hipError_t zero_two(float* a, int64_t na, float* b, int64_t nb, hipStream_t s) {
  const int64_t n = na + nb;
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(zero_two_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a, na, b, nb);
  return hipGetLastError();
}

// Decay-gradient partial rows the memory backward writes in a call (with or
// without carried state), and the most any call writes.
int dg_part_rows_used(int B, int nb, int D, bool per_channel, bool carry) {
  if (mem_fused(nb, per_channel))
    return per_channel ? B : ((D + kMsCols - 1) / kMsCols) * B;
  const int ns = lb_nseg(B, nb, D, per_channel, carry);
  if (ns) return B * ((D + kScCols - 1) / kScCols) * ns;
  return per_channel ? B : ((D + kScCols - 1) / kScCols) * B;
}

int dg_part_rows(int B, int nb, int D, bool per_channel) {
  return std::max(dg_part_rows_used(B, nb, D, per_channel, false),
                  dg_part_rows_used(B, nb, D, per_channel, true));
}

hipError_t dgamma_reduce(const float* part, int rows, int Dp, float* out, bool accumulate,
                         hipStream_t s) {
  if (!out) return hipSuccess;
  hipLaunchKernelGGL(dgamma_reduce_kernel, dim3(Dp == 1 ? 1 : (Dp + 63) / 64), dim3(256), 0, s,
                     part, rows, Dp, out, accumulate ? 1 : 0);
  return hipGetLastError();
}

hipError_t fill_f32(float* p, int64_t n, float v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(fill_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

}  // namespace bcmt
