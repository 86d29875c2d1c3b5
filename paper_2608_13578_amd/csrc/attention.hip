// Block-local causal multi-head attention (Sec. 3.3 and 3.6 of the paper):
// for every batch element, block and head, softmax(Q K^T / sqrt(dh) + causal
// mask) V over the block's own tokens, the diagonal included.  No score
// matrix ever leaves registers: the softmax is evaluated online over 64-key
// tiles staged in LDS, and the forward keeps only a per-query log-sum-exp for
// the backward recomputation.
//
// Head width is 64.  Work decomposition (one workgroup per (query or key
// tile, block, batch * head)); each wave owns 32 queries (forward and dQ) or
// 32 keys (dK/dV) as two 16-wide sub-tiles.
//
// Register layouts (see common.h): a matrix instruction returns lane l the
// column (l % 16) and rows 4*(l/16) + r, r = 0..3.  The forward computes the
// transposed scores S^T[u][t] = K[u] . Q[t], so that a lane holds one query t
// = l % 16 and a set of keys.  Those probabilities are then directly the
// second operand of O^T[d][t] = sum_u V^T[d][u] P^T[u][t]: the eight K
// elements lane group g contributes are the keys 4g..4g+3 and 16+4g..16+4g+3
// of a 32-key step, and the V^T operand is read from LDS with the same key
// order.  Because every lane keeps one query throughout, the running max and
// sum of the online softmax never move between lanes except for the final
// reduction over the four lane groups.
#include "common.h"
#include "kernels.h"

namespace bcmt {
namespace {

constexpr int kDh = 64;

template <typename T> struct AttnLds {
  static constexpr int VE = Vec16<T>::N;
  static constexpr int NAT = kDh + VE;  // row of a natural [row][d] tile
  static constexpr int TR = kDh + 4;    // row of a transposed [d][row] tile
};

// Stage rows r0 .. r0+63 (clipped at rmax) of a 64-column slice into LDS,
// natural and/or transposed.  Rows past rmax are zero, so that no stale LDS
// value ever meets a zero probability in a product.
template <typename T, bool NAT, bool TRN>
__device__ __forceinline__ void stage_tile(const T* src, int64_t rs, int r0, int rmax, T* nat,
                                           T* trn, int tid, int nthr) {
  constexpr int VE = Vec16<T>::N;
  constexpr int VPR = kDh / VE;
  typedef typename Vec16<T>::type vec;
  for (int idx = tid; idx < 64 * VPR; idx += nthr) {
    const int r = idx / VPR;
    const int c = (idx % VPR) * VE;
    const int row = r0 + r;
    vec v = row < rmax ? load16(src + (int64_t)row * rs + c) : vec{};
    if constexpr (NAT) store16(nat + r * AttnLds<T>::NAT + c, v);
    if constexpr (TRN) {
#pragma unroll
      for (int e = 0; e < VE; ++e) trn[(c + e) * AttnLds<T>::TR + r] = v[e];
    }
  }
}

template <typename T>
__device__ __forceinline__ typename Frag<T>::type frag_global(const T* p, bool ok) {
  typedef typename Frag<T>::type F;
  return ok ? load_frag(p) : F{};
}

// ------------------------------------------------------------------ forward

template <typename T>
__global__ __launch_bounds__(256) void attn_fwd_kernel(const T* __restrict__ qkv,
                                                       T* __restrict__ out,
                                                       float* __restrict__ lse, int Tn, int D,
                                                       int H, int L, float sl2) {
  typedef typename Frag<T>::type F;
  constexpr int NAT = AttnLds<T>::NAT, TR = AttnLds<T>::TR;
  __shared__ __attribute__((aligned(16))) T Ks[64 * NAT];
  __shared__ __attribute__((aligned(16))) T Vt[64 * TR];

  const int nthr = blockDim.x;
  const int QT = (nthr / 64) * 32;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int b = blockIdx.z / H, h = blockIdx.z % H;
  const int bs = blockIdx.y * L;
  const int be = min(bs + L, Tn);
  const int q0 = bs + blockIdx.x * QT;
  if (q0 >= be) return;
  const int64_t rs = 3LL * D;
  const T* base = qkv + (int64_t)b * Tn * rs + h * kDh;
  const int tw0 = q0 + wave * 32;

  F qf[2][2];
#pragma unroll
  for (int nq = 0; nq < 2; ++nq) {
    const int t = tw0 + nq * 16 + lr;
#pragma unroll
    for (int ds = 0; ds < 2; ++ds)
      qf[nq][ds] = frag_global(base + (int64_t)t * rs + ds * 32 + lg * 8, t < be);
  }
  f32x4 o[2][4];
  float m[2], l[2];
#pragma unroll
  for (int nq = 0; nq < 2; ++nq) {
    m[nq] = -INFINITY;
    l[nq] = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) o[nq][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  const int kend = min(be, q0 + QT);
  for (int kt = bs; kt < kend; kt += 64) {
    __syncthreads();
    stage_tile<T, true, false>(base + D, rs, kt, kend, Ks, nullptr, tid, nthr);
    stage_tile<T, false, true>(base + 2 * D, rs, kt, kend, nullptr, Vt, tid, nthr);
    __syncthreads();
#pragma unroll
    for (int nq = 0; nq < 2; ++nq) {
      const int tq = tw0 + nq * 16;
      if (tq >= be || tq + 15 < kt) continue;  // wave-uniform
      f32x4 s[4];
#pragma unroll
      for (int ku = 0; ku < 4; ++ku) {
        s[ku] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ds = 0; ds < 2; ++ds)
          s[ku] = mma16(load_frag(Ks + (ku * 16 + lr) * NAT + ds * 32 + lg * 8), qf[nq][ds], s[ku]);
      }
      const int t_eff = min(tq + lr, be - 1);
      float mx = -INFINITY;
#pragma unroll
      for (int ku = 0; ku < 4; ++ku)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int u = kt + ku * 16 + lg * 4 + r;
          const float z = u <= t_eff ? s[ku][r] * sl2 : -INFINITY;
          s[ku][r] = z;
          mx = fmaxf(mx, z);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mnew = fmaxf(m[nq], mx);
      const float alpha = exp2f(m[nq] - mnew);
      float ps = 0.f;
#pragma unroll
      for (int ku = 0; ku < 4; ++ku)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = exp2f(s[ku][r] - mnew);
          s[ku][r] = p;
          ps += p;
        }
      l[nq] = l[nq] * alpha + ps;
      m[nq] = mnew;
#pragma unroll
      for (int j = 0; j < 4; ++j) o[nq][j] *= alpha;
#pragma unroll
      for (int us = 0; us < 2; ++us) {
        const F pf = frag_from<T>(s[2 * us], s[2 * us + 1]);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const T* vp = Vt + (j * 16 + lr) * TR + us * 32 + lg * 4;
          o[nq][j] = mma16(load_frag_split(vp, vp + 16), pf, o[nq][j]);
        }
      }
    }
  }

#pragma unroll
  for (int nq = 0; nq < 2; ++nq) {
    float lt = l[nq];
    lt += __shfl_xor(lt, 16, 64);
    lt += __shfl_xor(lt, 32, 64);
    const int t = tw0 + nq * 16 + lr;
    if (t < be) {
      const float inv = 1.0f / lt;
      T* op = out + ((int64_t)b * Tn + t) * D + h * kDh + lg * 4;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        store4(op + j * 16, o[nq][j][0] * inv, o[nq][j][1] * inv, o[nq][j][2] * inv,
               o[nq][j][3] * inv);
      if (lg == 0) lse[((int64_t)b * H + h) * Tn + t] = m[nq] + log2f(lt);
    }
  }
}

// ------------------------------------------------------------------ backward: dQ
// Recomputes S^T and dP^T = V dO^T per key tile, forms dZ^T = P^T (dP^T -
// delta) and accumulates dQ^T[d][t] = sum_u K^T[d][u] dZ^T[u][t].  Also
// produces delta_t = dO_t . O_t, which the dK/dV pass reads.

template <typename T>
__global__ __launch_bounds__(256) void attn_bwd_dq_kernel(
    const T* __restrict__ qkv, const T* __restrict__ o, const T* __restrict__ dout,
    const float* __restrict__ lse, float* __restrict__ delta, T* __restrict__ dqkv, int Tn,
    int D, int H, int L, float sl2, float scale) {
  typedef typename Frag<T>::type F;
  constexpr int NAT = AttnLds<T>::NAT, TR = AttnLds<T>::TR;
  __shared__ __attribute__((aligned(16))) T Ks[64 * NAT];
  __shared__ __attribute__((aligned(16))) T Kt[64 * TR];
  __shared__ __attribute__((aligned(16))) T Vs[64 * NAT];

  const int nthr = blockDim.x;
  const int QT = (nthr / 64) * 32;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int b = blockIdx.z / H, h = blockIdx.z % H;
  const int bs = blockIdx.y * L;
  const int be = min(bs + L, Tn);
  const int q0 = bs + blockIdx.x * QT;
  if (q0 >= be) return;
  const int64_t rs = 3LL * D;
  const T* base = qkv + (int64_t)b * Tn * rs + h * kDh;
  const T* ob = o + (int64_t)b * Tn * D + h * kDh;
  const T* db = dout + (int64_t)b * Tn * D + h * kDh;
  const int64_t lrow = ((int64_t)b * H + h) * Tn;
  const int tw0 = q0 + wave * 32;

  F qf[2][2], df[2][2];
  float dl[2], ls[2];
#pragma unroll
  for (int nq = 0; nq < 2; ++nq) {
    const int t = tw0 + nq * 16 + lr;
    const bool ok = t < be;
    float part = 0.f;
#pragma unroll
    for (int ds = 0; ds < 2; ++ds) {
      qf[nq][ds] = frag_global(base + (int64_t)t * rs + ds * 32 + lg * 8, ok);
      df[nq][ds] = frag_global(db + (int64_t)t * D + ds * 32 + lg * 8, ok);
      const F of = frag_global(ob + (int64_t)t * D + ds * 32 + lg * 8, ok);
#pragma unroll
      for (int e = 0; e < 8; ++e) part += to_f32(df[nq][ds][e]) * to_f32(of[e]);
    }
    part += __shfl_xor(part, 16, 64);
    part += __shfl_xor(part, 32, 64);
    dl[nq] = part;
    ls[nq] = ok ? lse[lrow + t] : 0.f;
    if (ok && lg == 0) delta[lrow + t] = part;
  }
  f32x4 dq[2][4];
#pragma unroll
  for (int nq = 0; nq < 2; ++nq)
#pragma unroll
    for (int j = 0; j < 4; ++j) dq[nq][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int kend = min(be, q0 + QT);
  for (int kt = bs; kt < kend; kt += 64) {
    __syncthreads();
    stage_tile<T, true, true>(base + D, rs, kt, kend, Ks, Kt, tid, nthr);
    stage_tile<T, true, false>(base + 2 * D, rs, kt, kend, Vs, nullptr, tid, nthr);
    __syncthreads();
#pragma unroll
    for (int nq = 0; nq < 2; ++nq) {
      const int tq = tw0 + nq * 16;
      if (tq >= be || tq + 15 < kt) continue;  // wave-uniform
      f32x4 s[4], dp[4];
#pragma unroll
      for (int ku = 0; ku < 4; ++ku) {
        s[ku] = f32x4{0.f, 0.f, 0.f, 0.f};
        dp[ku] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ds = 0; ds < 2; ++ds) {
          s[ku] = mma16(load_frag(Ks + (ku * 16 + lr) * NAT + ds * 32 + lg * 8), qf[nq][ds], s[ku]);
          dp[ku] = mma16(load_frag(Vs + (ku * 16 + lr) * NAT + ds * 32 + lg * 8), df[nq][ds], dp[ku]);
        }
      }
      const int t_eff = min(tq + lr, be - 1);
#pragma unroll
      for (int ku = 0; ku < 4; ++ku)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int u = kt + ku * 16 + lg * 4 + r;
          const float p = u <= t_eff ? exp2f(s[ku][r] * sl2 - ls[nq]) : 0.f;
          s[ku][r] = p * (dp[ku][r] - dl[nq]);
        }
#pragma unroll
      for (int us = 0; us < 2; ++us) {
        const F zf = frag_from<T>(s[2 * us], s[2 * us + 1]);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const T* kp = Kt + (j * 16 + lr) * TR + us * 32 + lg * 4;
          dq[nq][j] = mma16(load_frag_split(kp, kp + 16), zf, dq[nq][j]);
        }
      }
    }
  }

#pragma unroll
  for (int nq = 0; nq < 2; ++nq) {
    const int t = tw0 + nq * 16 + lr;
    if (t < be) {
      T* p = dqkv + ((int64_t)b * Tn + t) * rs + h * kDh + lg * 4;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        store4(p + j * 16, dq[nq][j][0] * scale, dq[nq][j][1] * scale, dq[nq][j][2] * scale,
               dq[nq][j][3] * scale);
    }
  }
}

// ------------------------------------------------------------------ backward: dK, dV
// Each wave keeps its 32 keys' K and V fragments in registers and walks the
// query tiles at or after them: S[t][u] and dP[t][u] land with one key per
// lane, and dV^T[d][u] += sum_t dO^T[d][t] P[t][u], dK^T[d][u] += sum_t
// Q^T[d][t] dZ[t][u] take those registers directly as their second operand.

template <typename T>
__global__ __launch_bounds__(256) void attn_bwd_dkdv_kernel(
    const T* __restrict__ qkv, const T* __restrict__ dout, const float* __restrict__ lse,
    const float* __restrict__ delta, T* __restrict__ dqkv, int Tn, int D, int H, int L,
    float sl2, float scale) {
  typedef typename Frag<T>::type F;
  constexpr int NAT = AttnLds<T>::NAT, TR = AttnLds<T>::TR;
  __shared__ __attribute__((aligned(16))) T Qs[64 * NAT];
  __shared__ __attribute__((aligned(16))) T Qt[64 * TR];
  __shared__ __attribute__((aligned(16))) T Ds[64 * NAT];
  __shared__ __attribute__((aligned(16))) T Dt[64 * TR];
  __shared__ float ls_s[64];
  __shared__ float dl_s[64];

  const int nthr = blockDim.x;
  const int KT = (nthr / 64) * 32;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int b = blockIdx.z / H, h = blockIdx.z % H;
  const int bs = blockIdx.y * L;
  const int be = min(bs + L, Tn);
  const int k0 = bs + blockIdx.x * KT;
  if (k0 >= be) return;
  const int64_t rs = 3LL * D;
  const T* base = qkv + (int64_t)b * Tn * rs + h * kDh;
  const T* db = dout + (int64_t)b * Tn * D + h * kDh;
  const int64_t lrow = ((int64_t)b * H + h) * Tn;
  const int uw0 = k0 + wave * 32;

  F kf[2][2], vf[2][2];
#pragma unroll
  for (int ku = 0; ku < 2; ++ku) {
    const int u = uw0 + ku * 16 + lr;
#pragma unroll
    for (int ds = 0; ds < 2; ++ds) {
      kf[ku][ds] = frag_global(base + D + (int64_t)u * rs + ds * 32 + lg * 8, u < be);
      vf[ku][ds] = frag_global(base + 2 * D + (int64_t)u * rs + ds * 32 + lg * 8, u < be);
    }
  }
  f32x4 dk[2][4], dv[2][4];
#pragma unroll
  for (int ku = 0; ku < 2; ++ku)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      dk[ku][j] = f32x4{0.f, 0.f, 0.f, 0.f};
      dv[ku][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

  for (int tt = k0; tt < be; tt += 64) {
    __syncthreads();
    stage_tile<T, true, true>(base, rs, tt, be, Qs, Qt, tid, nthr);
    stage_tile<T, true, true>(db, D, tt, be, Ds, Dt, tid, nthr);
    for (int i = tid; i < 64; i += nthr) {
      const int t = tt + i;
      ls_s[i] = t < be ? lse[lrow + t] : 0.f;
      dl_s[i] = t < be ? delta[lrow + t] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int ku = 0; ku < 2; ++ku) {
      const int uw = uw0 + ku * 16;
      if (uw >= be || tt + 63 < uw) continue;  // wave-uniform
      const int u = uw + lr;
      f32x4 p[4], z[4];
#pragma unroll
      for (int ts = 0; ts < 4; ++ts) {
        f32x4 s = {0.f, 0.f, 0.f, 0.f}, dp = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ds = 0; ds < 2; ++ds) {
          s = mma16(load_frag(Qs + (ts * 16 + lr) * NAT + ds * 32 + lg * 8), kf[ku][ds], s);
          dp = mma16(load_frag(Ds + (ts * 16 + lr) * NAT + ds * 32 + lg * 8), vf[ku][ds], dp);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int ti = ts * 16 + lg * 4 + r;
          const int t = tt + ti;
          const bool ok = t >= u && t < be && u < be;
          const float pv = ok ? exp2f(s[r] * sl2 - ls_s[ti]) : 0.f;
          p[ts][r] = pv;
          z[ts][r] = pv * (dp[r] - dl_s[ti]);
        }
      }
#pragma unroll
      for (int tq = 0; tq < 2; ++tq) {
        const F pf = frag_from<T>(p[2 * tq], p[2 * tq + 1]);
        const F zf = frag_from<T>(z[2 * tq], z[2 * tq + 1]);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const T* dp_ = Dt + (j * 16 + lr) * TR + tq * 32 + lg * 4;
          dv[ku][j] = mma16(load_frag_split(dp_, dp_ + 16), pf, dv[ku][j]);
          const T* qp = Qt + (j * 16 + lr) * TR + tq * 32 + lg * 4;
          dk[ku][j] = mma16(load_frag_split(qp, qp + 16), zf, dk[ku][j]);
        }
      }
    }
  }

#pragma unroll
  for (int ku = 0; ku < 2; ++ku) {
    const int u = uw0 + ku * 16 + lr;
    if (u < be) {
      T* p = dqkv + ((int64_t)b * Tn + u) * rs + h * kDh + lg * 4;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        store4(p + D + j * 16, dk[ku][j][0] * scale, dk[ku][j][1] * scale, dk[ku][j][2] * scale,
               dk[ku][j][3] * scale);
        store4(p + 2 * D + j * 16, dv[ku][j][0], dv[ku][j][1], dv[ku][j][2], dv[ku][j][3]);
      }
    }
  }
}

// ------------------------------------------------------------------ bf16 kernels
// The bf16 path stages every 64 x 64 tile in its natural [row][d] layout
// with direct global->LDS loads (double buffered), and reads the transposed
// operands (V^T for P V, K^T for dQ, Q^T and dO^T for dK and dV) from the
// same tiles with ds_read_b64_tr_b16: within each 16-lane group, lane i gets
// element (i % 4) of the 4-element rows addressed by lanes 4j + i/4; with
// lane q addressing row k0 + q/4 at column c0 + 4 (q % 4), lane i receives
// rows k0..k0+3 of column c0 + i.  Tile element (r, c) lives at
// r*64 + 8*((c/8) ^ tswz(r)) + c % 8.  A row read (16 lanes, 16 consecutive
// rows, one chunk) needs rows 2j and 2j+1 (the two halves of the 64 banks)
// on distinct chunks for distinct j: tswz is a permutation of the bits of
// r/2.  A transposing read (16 lanes, 4 consecutive rows from a multiple of
// 4, two adjacent chunks) needs rows 4j and 4j+2 on disjoint chunk pairs,
// so row bit 1 goes to chunk bit 1; the next lane group (row bit 2, or row
// bit 3 in tcol8p's order) moves to the other pairs through chunk bit 2.
// (The plain (r/2) % 8 put rows 4j and 4j+2 on the same chunks: a two-way
// conflict on every transposing read.)
__device__ __forceinline__ int tswz(int r) {
  return ((r >> 3) & 1) | (r & 2) | (((r ^ (r >> 1)) & 4));
}
__device__ __forceinline__ int toff(int r, int c) {
  return r * 64 + (((c >> 3) ^ tswz(r)) << 3) + (c & 7);
}
__device__ __forceinline__ bf16x8 trow8(const bf16* t, int r, int c0) {
  return *reinterpret_cast<const bf16x8*>(t + toff(r, c0));
}
// The same through inline assembly (see lds_read_tr()).
__device__ __forceinline__ bf16x8 trow8a(const bf16* t, int r, int c0) {
  return lds_read_b128(t + toff(r, c0));
}
__device__ __forceinline__ bf16x4 tcol4(const bf16* t, int k0, int c0, int lane) {
  const int i = lane & 15;
  return lds_read_tr(t + toff(k0 + (i >> 2), c0 + ((i & 3) << 2)));
}
// Operand over d (rows dsub*16 + lane%16) and the 32 keys/queries
// {b0 + 4g .. +3} u {b0 + 16 + 4g .. +3} of lane group g: the order in which
// a transposed-score tile holds its probabilities.
__device__ __forceinline__ bf16x8 tcol8p(const bf16* t, int b0, int dsub, int lane) {
  const int g = lane >> 4;
  const bf16x4 a = tcol4(t, b0 + 4 * g, dsub * 16, lane);
  const bf16x4 b = tcol4(t, b0 + 16 + 4 * g, dsub * 16, lane);
  bf16x8 r = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  return r;
}

// This wave's direct loads of a 64 x 64 tile: rows r0 .. r0+63 of `src`
// (row stride rs), clamped to rlast (clamped rows are never used unmasked).
template <int NW>
__device__ __forceinline__ void tile_issue(const bf16* src, int64_t rs, int r0, int rlast,
                                           bf16* t, int wave, int lane) {
#pragma unroll
  for (int i = 0; i < 8 / NW; ++i) {
    const int gi = wave * (8 / NW) + i;
    const int row = gi * 8 + (lane >> 3);
    const int cg = (lane & 7) ^ tswz(row);
    const int grow = min(r0 + row, rlast);
    __builtin_amdgcn_global_load_lds(src + (int64_t)grow * rs + cg * 8, (lds_void_t*)(t + gi * 512),
                                     16, 0, 0);
  }
}
// 64 floats (one per lane of wave 0), indices clamped to last.
__device__ __forceinline__ void vec_issue(const float* src, int i0, int last, float* dst, int lane) {
  __builtin_amdgcn_global_load_lds(src + min(i0 + lane, last), (lds_void_t*)dst, 4, 0, 0);
}

template <int N>
__device__ __forceinline__ void vm_wait() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
__device__ __forceinline__ void sync_lds() {
  __builtin_amdgcn_s_barrier();
}

template <int NW>
__global__ __launch_bounds__(NW * 64, 3) void attn_fwd_bf16_kernel(const bf16* __restrict__ qkv,
                                                               bf16* __restrict__ out,
                                                               float* __restrict__ lse, int Tn,
                                                               int D, int H, int L, float sl2) {
  constexpr int QT = NW * 32;
  constexpr int NI = 16 / NW;  // direct loads per wave per key tile (K and V)
  __shared__ __attribute__((aligned(1024))) bf16 lds[2][2][64 * 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int b = blockIdx.z / H, h = blockIdx.z % H;
  const int bs = blockIdx.y * L;
  const int be = min(bs + L, Tn);
  const int q0 = bs + blockIdx.x * QT;
  if (q0 >= be) return;
  const int64_t rs = 3LL * D;
  const bf16* base = qkv + (int64_t)b * Tn * rs + h * kDh;
  // The workgroup's 2 NW groups of 16 queries are dealt in pairs g, 2 NW - 1 - g,
  // one pair per wave: a causal group's work grows with its position, so
  // every wave gets about the same number of (query group, key tile) pairs.
  const int tq[2] = {q0 + 16 * wave, q0 + 16 * (2 * NW - 1 - wave)};
  const int kend = min(be, q0 + QT);
  const int nt = (kend - bs + 63) / 64;

  bf16x8 qf[2][2];
#pragma unroll
  for (int nq = 0; nq < 2; ++nq) {
    const int t = tq[nq] + lr;
#pragma unroll
    for (int ds = 0; ds < 2; ++ds)
      qf[nq][ds] = t < be ? *reinterpret_cast<const bf16x8*>(base + (int64_t)t * rs + ds * 32 + lg * 8)
                          : bf16x8{};
  }
  f32x4 o[2][4];
  float m[2], l[2];
#pragma unroll
  for (int nq = 0; nq < 2; ++nq) {
    m[nq] = -INFINITY;
    l[nq] = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) o[nq][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  tile_issue<NW>(base + D, rs, bs, kend - 1, lds[0][0], wave, lane);
  tile_issue<NW>(base + 2 * D, rs, bs, kend - 1, lds[0][1], wave, lane);
  if (nt > 1) {
    tile_issue<NW>(base + D, rs, bs + 64, kend - 1, lds[1][0], wave, lane);
    tile_issue<NW>(base + 2 * D, rs, bs + 64, kend - 1, lds[1][1], wave, lane);
  }
  for (int it = 0; it < nt; ++it) {
    if (it + 1 < nt) vm_wait<NI>();
    else vm_wait<0>();
    sync_lds();
    const int kt = bs + it * 64;
    const bf16* Kt = lds[it & 1][0];
    const bf16* Vt = lds[it & 1][1];
    // Scores of both query groups first (the key fragments are dead after
    // that), then the softmax update, then the value fragments and P V: at
    // most one of the two fragment sets is live at a time.  (Every wave
    // still reaches the barriers below.)
    bool live[2];
#pragma unroll
    for (int nq = 0; nq < 2; ++nq) {
      live[nq] = !(tq[nq] >= be || tq[nq] + 15 < kt);  // wave-uniform
    }
    f32x4 s[2][4];
    if (live[0] || live[1]) {
      bf16x8 kf[4][2];
#pragma unroll
      for (int ku = 0; ku < 4; ++ku)
#pragma unroll
        for (int ds = 0; ds < 2; ++ds) kf[ku][ds] = trow8(Kt, ku * 16 + lr, ds * 32 + lg * 8);
#pragma unroll
      for (int nq = 0; nq < 2; ++nq)
#pragma unroll
        for (int ku = 0; ku < 4; ++ku) {
          s[nq][ku] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ds = 0; ds < 2; ++ds) s[nq][ku] = mma16(kf[ku][ds], qf[nq][ds], s[nq][ku]);
        }
    }
#pragma unroll
    for (int nq = 0; nq < 2; ++nq) {
      if (!live[nq]) continue;
      const int t_eff = min(tq[nq] + lr, be - 1);
      float mx = -INFINITY;
#pragma unroll
      for (int ku = 0; ku < 4; ++ku)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int u = kt + ku * 16 + lg * 4 + r;
          const float z = u <= t_eff ? s[nq][ku][r] * sl2 : -INFINITY;
          s[nq][ku][r] = z;
          mx = fmaxf(mx, z);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mnew = fmaxf(m[nq], mx);
      const float alpha = exp2_fast(m[nq] - mnew);
      float ps = 0.f;
#pragma unroll
      for (int ku = 0; ku < 4; ++ku)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float pv = exp2_fast(s[nq][ku][r] - mnew);
          s[nq][ku][r] = pv;
          ps += pv;
        }
      l[nq] = l[nq] * alpha + ps;
      m[nq] = mnew;
#pragma unroll
      for (int j = 0; j < 4; ++j) o[nq][j] *= alpha;
    }
    if (live[0] || live[1]) {
      bf16x8 vf[4][2];
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int us = 0; us < 2; ++us) vf[j][us] = tcol8p(Vt, us * 32, j, lane);
      lds_tr_wait();
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int us = 0; us < 2; ++us) lds_tr_bind(vf[j][us]);
#pragma unroll
      for (int nq = 0; nq < 2; ++nq) {
        if (!live[nq]) continue;
#pragma unroll
        for (int us = 0; us < 2; ++us) {
          const bf16x8 pf = frag_from<bf16>(s[nq][2 * us], s[nq][2 * us + 1]);
#pragma unroll
          for (int j = 0; j < 4; ++j) o[nq][j] = mma16(vf[j][us], pf, o[nq][j]);
        }
      }
    }
    if (it + 2 < nt) {
      sync_lds();  // every wave is done with this buffer
      tile_issue<NW>(base + D, rs, kt + 128, kend - 1, lds[it & 1][0], wave, lane);
      tile_issue<NW>(base + 2 * D, rs, kt + 128, kend - 1, lds[it & 1][1], wave, lane);
    }
  }

#pragma unroll
  for (int nq = 0; nq < 2; ++nq) {
    float lt = l[nq];
    lt += __shfl_xor(lt, 16, 64);
    lt += __shfl_xor(lt, 32, 64);
    const int t = tq[nq] + lr;
    if (t < be) {
      const float inv = 1.0f / lt;
      bf16* op = out + ((int64_t)b * Tn + t) * D + h * kDh + lg * 4;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        store4(op + j * 16, o[nq][j][0] * inv, o[nq][j][1] * inv, o[nq][j][2] * inv,
               o[nq][j][3] * inv);
      if (lg == 0) lse[((int64_t)b * H + h) * Tn + t] = m[nq] + log2f(lt);
    }
  }
}

template <int NW>
__global__ __launch_bounds__(NW * 64) void attn_bwd_dq_bf16_kernel(
    const bf16* __restrict__ qkv, const bf16* __restrict__ o, const bf16* __restrict__ dout,
    const float* __restrict__ lse, float* __restrict__ delta, bf16* __restrict__ dqkv, int Tn,
    int D, int H, int L, float sl2, float scale) {
  constexpr int QT = NW * 32;
  constexpr int NI = 16 / NW;
  __shared__ __attribute__((aligned(1024))) bf16 lds[2][2][64 * 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int b = blockIdx.z / H, h = blockIdx.z % H;
  const int bs = blockIdx.y * L;
  const int be = min(bs + L, Tn);
  const int q0 = bs + blockIdx.x * QT;
  if (q0 >= be) return;
  const int64_t rs = 3LL * D;
  const bf16* base = qkv + (int64_t)b * Tn * rs + h * kDh;
  const bf16* ob = o + (int64_t)b * Tn * D + h * kDh;
  const bf16* db = dout + (int64_t)b * Tn * D + h * kDh;
  const int64_t lrow = ((int64_t)b * H + h) * Tn;
  const int tw0 = q0 + wave * 32;
  const int kend = min(be, q0 + QT);
  const int nt = (kend - bs + 63) / 64;

  bf16x8 qf[2][2], df[2][2];
  float dl[2], ls[2];
#pragma unroll
  for (int nq = 0; nq < 2; ++nq) {
    const int t = tw0 + nq * 16 + lr;
    const bool ok = t < be;
    float part = 0.f;
#pragma unroll
    for (int ds = 0; ds < 2; ++ds) {
      qf[nq][ds] = ok ? *reinterpret_cast<const bf16x8*>(base + (int64_t)t * rs + ds * 32 + lg * 8) : bf16x8{};
      df[nq][ds] = ok ? *reinterpret_cast<const bf16x8*>(db + (int64_t)t * D + ds * 32 + lg * 8) : bf16x8{};
      const bf16x8 of = ok ? *reinterpret_cast<const bf16x8*>(ob + (int64_t)t * D + ds * 32 + lg * 8) : bf16x8{};
#pragma unroll
      for (int e = 0; e < 8; ++e) part += (float)df[nq][ds][e] * (float)of[e];
    }
    part += __shfl_xor(part, 16, 64);
    part += __shfl_xor(part, 32, 64);
    dl[nq] = part;
    ls[nq] = ok ? lse[lrow + t] : 0.f;
    if (ok && lg == 0) delta[lrow + t] = part;
  }
  f32x4 dq[2][4];
#pragma unroll
  for (int nq = 0; nq < 2; ++nq)
#pragma unroll
    for (int j = 0; j < 4; ++j) dq[nq][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  tile_issue<NW>(base + D, rs, bs, kend - 1, lds[0][0], wave, lane);
  tile_issue<NW>(base + 2 * D, rs, bs, kend - 1, lds[0][1], wave, lane);
  if (nt > 1) {
    tile_issue<NW>(base + D, rs, bs + 64, kend - 1, lds[1][0], wave, lane);
    tile_issue<NW>(base + 2 * D, rs, bs + 64, kend - 1, lds[1][1], wave, lane);
  }
  for (int it = 0; it < nt; ++it) {
    if (it + 1 < nt) vm_wait<NI>();
    else vm_wait<0>();
    sync_lds();
    const int kt = bs + it * 64;
    const bf16* Kt = lds[it & 1][0];
    const bf16* Vt = lds[it & 1][1];
    bf16x8 kf[4][2], vf[4][2], ktf[4][2];
#pragma unroll
    for (int ku = 0; ku < 4; ++ku)
#pragma unroll
      for (int ds = 0; ds < 2; ++ds) {
        kf[ku][ds] = trow8(Kt, ku * 16 + lr, ds * 32 + lg * 8);
        vf[ku][ds] = trow8(Vt, ku * 16 + lr, ds * 32 + lg * 8);
      }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int us = 0; us < 2; ++us) ktf[j][us] = tcol8p(Kt, us * 32, j, lane);
    lds_tr_wait();
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int us = 0; us < 2; ++us) lds_tr_bind(ktf[j][us]);
#pragma unroll
    for (int nq = 0; nq < 2; ++nq) {
      const int tq = tw0 + nq * 16;
      if (tq >= be || tq + 15 < kt) continue;  // wave-uniform
      f32x4 s[4], dp[4];
#pragma unroll
      for (int ku = 0; ku < 4; ++ku) {
        s[ku] = f32x4{0.f, 0.f, 0.f, 0.f};
        dp[ku] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ds = 0; ds < 2; ++ds) {
          s[ku] = mma16(kf[ku][ds], qf[nq][ds], s[ku]);
          dp[ku] = mma16(vf[ku][ds], df[nq][ds], dp[ku]);
        }
      }
      const int t_eff = min(tq + lr, be - 1);
#pragma unroll
      for (int ku = 0; ku < 4; ++ku)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int u = kt + ku * 16 + lg * 4 + r;
          const float pv = u <= t_eff ? exp2_fast(s[ku][r] * sl2 - ls[nq]) : 0.f;
          s[ku][r] = pv * (dp[ku][r] - dl[nq]);
        }
#pragma unroll
      for (int us = 0; us < 2; ++us) {
        const bf16x8 zf = frag_from<bf16>(s[2 * us], s[2 * us + 1]);
#pragma unroll
        for (int j = 0; j < 4; ++j) dq[nq][j] = mma16(ktf[j][us], zf, dq[nq][j]);
      }
    }
    if (it + 2 < nt) {
      sync_lds();
      tile_issue<NW>(base + D, rs, kt + 128, kend - 1, lds[it & 1][0], wave, lane);
      tile_issue<NW>(base + 2 * D, rs, kt + 128, kend - 1, lds[it & 1][1], wave, lane);
    }
  }

#pragma unroll
  for (int nq = 0; nq < 2; ++nq) {
    const int t = tw0 + nq * 16 + lr;
    if (t < be) {
      bf16* p = dqkv + ((int64_t)b * Tn + t) * rs + h * kDh + lg * 4;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        store4(p + j * 16, dq[nq][j][0] * scale, dq[nq][j][1] * scale, dq[nq][j][2] * scale,
               dq[nq][j][3] * scale);
    }
  }
}

template <int NW>
__global__ __launch_bounds__(NW * 64) void attn_bwd_dkdv_bf16_kernel(
    const bf16* __restrict__ qkv, const bf16* __restrict__ dout, const float* __restrict__ lse,
    const float* __restrict__ delta, bf16* __restrict__ dqkv, int Tn, int D, int H, int L,
    float sl2, float scale) {
  constexpr int KT = NW * 32;
  constexpr int NI = 16 / NW;
  __shared__ __attribute__((aligned(1024))) bf16 lds[2][2][64 * 64];
  __shared__ __attribute__((aligned(16))) float vec_s[2][2][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int b = blockIdx.z / H, h = blockIdx.z % H;
  const int bs = blockIdx.y * L;
  const int be = min(bs + L, Tn);
  const int k0 = bs + blockIdx.x * KT;
  if (k0 >= be) return;
  const int64_t rs = 3LL * D;
  const bf16* base = qkv + (int64_t)b * Tn * rs + h * kDh;
  const bf16* db = dout + (int64_t)b * Tn * D + h * kDh;
  const int64_t lrow = ((int64_t)b * H + h) * Tn;
  const int uw0 = k0 + wave * 32;
  const int nt = (be - k0 + 63) / 64;

  bf16x8 kf[2][2], vf[2][2];
#pragma unroll
  for (int ku = 0; ku < 2; ++ku) {
    const int u = uw0 + ku * 16 + lr;
#pragma unroll
    for (int ds = 0; ds < 2; ++ds) {
      kf[ku][ds] = u < be ? *reinterpret_cast<const bf16x8*>(base + D + (int64_t)u * rs + ds * 32 + lg * 8) : bf16x8{};
      vf[ku][ds] = u < be ? *reinterpret_cast<const bf16x8*>(base + 2 * D + (int64_t)u * rs + ds * 32 + lg * 8) : bf16x8{};
    }
  }
  f32x4 dk[2][4], dv[2][4];
#pragma unroll
  for (int ku = 0; ku < 2; ++ku)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      dk[ku][j] = f32x4{0.f, 0.f, 0.f, 0.f};
      dv[ku][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

  auto issue = [&](int tt, int buf) {
    tile_issue<NW>(base, rs, tt, be - 1, lds[buf][0], wave, lane);
    tile_issue<NW>(db, D, tt, be - 1, lds[buf][1], wave, lane);
    if (wave == 0) {
      vec_issue(lse + lrow, tt, be - 1, vec_s[buf][0], lane);
      vec_issue(delta + lrow, tt, be - 1, vec_s[buf][1], lane);
    }
  };
  issue(k0, 0);
  if (nt > 1) issue(k0 + 64, 1);
  for (int it = 0; it < nt; ++it) {
    if (it + 1 < nt) {
      if (wave == 0) vm_wait<NI + 2>();
      else vm_wait<NI>();
    } else {
      vm_wait<0>();
    }
    sync_lds();
    const int tt = k0 + it * 64;
    const bf16* Qt = lds[it & 1][0];
    const bf16* Dt = lds[it & 1][1];
    // This lane's 16 queries of the tile: ts * 16 + lg * 4 + r.
    f32x4 lsv[4], dlv[4];
#pragma unroll
    for (int ts = 0; ts < 4; ++ts) {
      lsv[ts] = lds_read_f32x4(&vec_s[it & 1][0][ts * 16 + lg * 4]);
      dlv[ts] = lds_read_f32x4(&vec_s[it & 1][1][ts * 16 + lg * 4]);
    }
    lds_tr_wait();
#pragma unroll
    for (int ts = 0; ts < 4; ++ts) {
      lds_tr_bind(lsv[ts]);
      lds_tr_bind(dlv[ts]);
    }
#pragma unroll
    for (int ku = 0; ku < 2; ++ku) {
      const int uw = uw0 + ku * 16;
      if (uw >= be || tt + 63 < uw) continue;  // wave-uniform
      const int u = uw + lr;
      f32x4 p[4], z[4];
#pragma unroll
      for (int ts = 0; ts < 4; ++ts) {
        f32x4 s = {0.f, 0.f, 0.f, 0.f}, dp = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ds = 0; ds < 2; ++ds) {
          s = mma16(trow8(Qt, ts * 16 + lr, ds * 32 + lg * 8), kf[ku][ds], s);
          dp = mma16(trow8(Dt, ts * 16 + lr, ds * 32 + lg * 8), vf[ku][ds], dp);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int ti = ts * 16 + lg * 4 + r;
          const int t = tt + ti;
          const bool ok = t >= u && t < be && u < be;
          const float pv = ok ? exp2_fast(s[r] * sl2 - lsv[ts][r]) : 0.f;
          p[ts][r] = pv;
          z[ts][r] = pv * (dp[r] - dlv[ts][r]);
        }
      }
#pragma unroll
      for (int tq = 0; tq < 2; ++tq) {
        const bf16x8 pf = frag_from<bf16>(p[2 * tq], p[2 * tq + 1]);
        const bf16x8 zf = frag_from<bf16>(z[2 * tq], z[2 * tq + 1]);
        bf16x8 dtf[4], qtf[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          dtf[j] = tcol8p(Dt, tq * 32, j, lane);
          qtf[j] = tcol8p(Qt, tq * 32, j, lane);
        }
        lds_tr_wait();
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          lds_tr_bind(dtf[j]);
          lds_tr_bind(qtf[j]);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          dv[ku][j] = mma16(dtf[j], pf, dv[ku][j]);
          dk[ku][j] = mma16(qtf[j], zf, dk[ku][j]);
        }
      }
    }
    if (it + 2 < nt) {
      sync_lds();
      issue(tt + 128, it & 1);
    }
  }

#pragma unroll
  for (int ku = 0; ku < 2; ++ku) {
    const int u = uw0 + ku * 16 + lr;
    if (u < be) {
      bf16* p = dqkv + ((int64_t)b * Tn + u) * rs + h * kDh + lg * 4;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        store4(p + D + j * 16, dk[ku][j][0] * scale, dk[ku][j][1] * scale, dk[ku][j][2] * scale,
               dk[ku][j][3] * scale);
        store4(p + 2 * D + j * 16, dv[ku][j][0], dv[ku][j][1], dv[ku][j][2], dv[ku][j][3]);
      }
    }
  }
}

// The two phases of the fused backward of one block, with the block's Q, K,
// V and dO in LDS as tiles of 64 rows (tile t of matrix m at
// blk + (m * NT + t) * 4096, m = Q, K, V, dO) and the lse and delta of its
// queries in ls / dl (block-relative).  `dst` is dqkv at the sequence's first
// row and the head's first column.

// dK, dV for keys bs + w0 .. +31: scores held transposed, as in
// attn_bwd_dkdv_bf16_kernel; key rows past the block end are masked to zero
// probability.  Query tiles are taken in halves of 32 rows: both 16-key
// groups share every fragment read of a half.  MASK = false serves the tiles
// whose every query follows every key of the wave, inside the block.
template <int NT, bool MASK>
__device__ __forceinline__ void blk_dkdv_tile(const bf16* Qt, const bf16* Dt, const float* lst,
                                              const float* dlt, const bf16x8 (&kf)[2][2],
                                              const bf16x8 (&vf)[2][2], f32x4 (&dk)[2][4],
                                              f32x4 (&dv)[2][4], int tt, int u0, int be,
                                              float sl2, int lane) {
  const int lr = lane & 15, lg = lane >> 4;
#pragma unroll
  for (int tq = 0; tq < 2; ++tq) {
    bf16x8 qr[2][2], dr[2][2], dtf[4], qtf[4];
    f32x4 lsv[2], dlv[2];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int ts = 2 * tq + hh;
#pragma unroll
      for (int ds = 0; ds < 2; ++ds) {
        qr[hh][ds] = trow8a(Qt, ts * 16 + lr, ds * 32 + lg * 8);
        dr[hh][ds] = trow8a(Dt, ts * 16 + lr, ds * 32 + lg * 8);
      }
      lsv[hh] = lds_read_f32x4(lst + ts * 16 + lg * 4);
      dlv[hh] = lds_read_f32x4(dlt + ts * 16 + lg * 4);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      dtf[j] = tcol8p(Dt, tq * 32, j, lane);
      qtf[j] = tcol8p(Qt, tq * 32, j, lane);
    }
    lds_tr_wait();
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
#pragma unroll
      for (int ds = 0; ds < 2; ++ds) {
        lds_tr_bind(qr[hh][ds]);
        lds_tr_bind(dr[hh][ds]);
      }
      lds_tr_bind(lsv[hh]);
      lds_tr_bind(dlv[hh]);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      lds_tr_bind(dtf[j]);
      lds_tr_bind(qtf[j]);
    }
    f32x4 p[2][2], z[2][2];  // [key group][query row group of the half]
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int ts = 2 * tq + hh;
#pragma unroll
      for (int ku = 0; ku < 2; ++ku) {
        f32x4 sc = {0.f, 0.f, 0.f, 0.f}, dp = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ds = 0; ds < 2; ++ds) {
          sc = mma16(qr[hh][ds], kf[ku][ds], sc);
          dp = mma16(dr[hh][ds], vf[ku][ds], dp);
        }
        const int u = u0 + ku * 16 + lr;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float pv = exp2_fast(sc[r] * sl2 - lsv[hh][r]);
          if (MASK) {
            const int t = tt + ts * 16 + lg * 4 + r;
            pv = (t >= u && t < be && u < be) ? pv : 0.f;
          }
          p[ku][hh][r] = pv;
          z[ku][hh][r] = pv * (dp[r] - dlv[hh][r]);
        }
      }
    }
#pragma unroll
    for (int ku = 0; ku < 2; ++ku) {
      const bf16x8 pf = frag_from<bf16>(p[ku][0], p[ku][1]);
      const bf16x8 zf = frag_from<bf16>(z[ku][0], z[ku][1]);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        dv[ku][j] = mma16(dtf[j], pf, dv[ku][j]);
        dk[ku][j] = mma16(qtf[j], zf, dk[ku][j]);
      }
    }
  }
}

template <int NT>
__device__ __forceinline__ void blk_dkdv(const bf16* blk, const float* ls, const float* dl,
                                         bf16* dst, int64_t rs, int D, int bs, int be, int w0,
                                         int ntile, float sl2, float scale, int lane) {
  const int lr = lane & 15, lg = lane >> 4;
  const int kt0 = w0 / 64, kr0 = w0 % 64;
  const bf16* Kb = blk + (1 * NT + kt0) * 4096;
  const bf16* Vb = blk + (2 * NT + kt0) * 4096;
  bf16x8 kf[2][2], vf[2][2];
#pragma unroll
  for (int ku = 0; ku < 2; ++ku)
#pragma unroll
    for (int ds = 0; ds < 2; ++ds) {
      kf[ku][ds] = trow8a(Kb, kr0 + ku * 16 + lr, ds * 32 + lg * 8);
      vf[ku][ds] = trow8a(Vb, kr0 + ku * 16 + lr, ds * 32 + lg * 8);
    }
  lds_tr_wait();
#pragma unroll
  for (int ku = 0; ku < 2; ++ku)
#pragma unroll
    for (int ds = 0; ds < 2; ++ds) {
      lds_tr_bind(kf[ku][ds]);
      lds_tr_bind(vf[ku][ds]);
    }
  f32x4 dk[2][4], dv[2][4];
#pragma unroll
  for (int ku = 0; ku < 2; ++ku)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      dk[ku][j] = f32x4{0.f, 0.f, 0.f, 0.f};
      dv[ku][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  const int u0 = bs + w0;
  for (int it = kt0; it < ntile; ++it) {
    const int tt = bs + it * 64;
    const bf16* Qt = blk + (0 * NT + it) * 4096;
    const bf16* Dt = blk + (3 * NT + it) * 4096;
    const bool full = tt >= u0 + 31 && tt + 63 < be && u0 + 31 < be;  // wave-uniform
    if (full)
      blk_dkdv_tile<NT, false>(Qt, Dt, ls + it * 64, dl + it * 64, kf, vf, dk, dv, tt, u0, be,
                               sl2, lane);
    else
      blk_dkdv_tile<NT, true>(Qt, Dt, ls + it * 64, dl + it * 64, kf, vf, dk, dv, tt, u0, be,
                              sl2, lane);
  }
#pragma unroll
  for (int ku = 0; ku < 2; ++ku) {
    const int u = u0 + ku * 16 + lr;
    if (u < be) {
      bf16* pp = dst + (int64_t)u * rs + lg * 4;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        store4(pp + D + j * 16, dk[ku][j][0] * scale, dk[ku][j][1] * scale, dk[ku][j][2] * scale,
               dk[ku][j][3] * scale);
        store4(pp + 2 * D + j * 16, dv[ku][j][0], dv[ku][j][1], dv[ku][j][2], dv[ku][j][3]);
      }
    }
  }
}

// dQ contribution of one key tile (keys kt ..) to 16 queries tq .. of this
// wave (as in attn_bwd_dq_bf16_kernel), recomputing the probabilities from
// lse.  MASK = false serves a tile whose every key precedes every query.
template <bool MASK>
__device__ __forceinline__ void blk_dq_group(const bf16x8 (&kf)[4][2], const bf16x8 (&vf)[4][2],
                                             const bf16x8 (&ktf)[4][2], const bf16x8 (&qf)[2],
                                             const bf16x8 (&df)[2], float ls, float dl,
                                             f32x4 (&dq)[4], int kt, int tq, int be, float sl2,
                                             int lane) {
  const int lr = lane & 15, lg = lane >> 4;
  f32x4 sc[4], dp[4];
#pragma unroll
  for (int ku = 0; ku < 4; ++ku) {
    sc[ku] = f32x4{0.f, 0.f, 0.f, 0.f};
    dp[ku] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ds = 0; ds < 2; ++ds) {
      sc[ku] = mma16(kf[ku][ds], qf[ds], sc[ku]);
      dp[ku] = mma16(vf[ku][ds], df[ds], dp[ku]);
    }
  }
  const int t_eff = min(tq + lr, be - 1);
#pragma unroll
  for (int ku = 0; ku < 4; ++ku)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float pv = exp2_fast(sc[ku][r] * sl2 - ls);
      if (MASK) pv = kt + ku * 16 + lg * 4 + r <= t_eff ? pv : 0.f;
      sc[ku][r] = pv * (dp[ku][r] - dl);
    }
#pragma unroll
  for (int us = 0; us < 2; ++us) {
    const bf16x8 zf = frag_from<bf16>(sc[2 * us], sc[2 * us + 1]);
#pragma unroll
    for (int j = 0; j < 4; ++j) dq[j] = mma16(ktf[j][us], zf, dq[j]);
  }
}

// dQ for queries bs + w0 .. +31.
template <int NT>
__device__ __forceinline__ void blk_dq(const bf16* blk, const float* ls_s, const float* dl_s,
                                       bf16* dst, int64_t rs, int bs, int be, int w0, float sl2,
                                       float scale, int lane) {
  const int lr = lane & 15, lg = lane >> 4;
  const int qt0 = w0 / 64, qr0 = w0 % 64;
  bf16x8 qf[2][2], df[2][2];
  float dl[2], ls[2];
#pragma unroll
  for (int nq = 0; nq < 2; ++nq) {
#pragma unroll
    for (int ds = 0; ds < 2; ++ds) {
      qf[nq][ds] = trow8a(blk + (0 * NT + qt0) * 4096, qr0 + nq * 16 + lr, ds * 32 + lg * 8);
      df[nq][ds] = trow8a(blk + (3 * NT + qt0) * 4096, qr0 + nq * 16 + lr, ds * 32 + lg * 8);
    }
    dl[nq] = lds_read_f32(dl_s + w0 + nq * 16 + lr);
    ls[nq] = lds_read_f32(ls_s + w0 + nq * 16 + lr);
  }
  lds_tr_wait();
#pragma unroll
  for (int nq = 0; nq < 2; ++nq) {
#pragma unroll
    for (int ds = 0; ds < 2; ++ds) {
      lds_tr_bind(qf[nq][ds]);
      lds_tr_bind(df[nq][ds]);
    }
    lds_tr_bind(dl[nq]);
    lds_tr_bind(ls[nq]);
  }
  f32x4 dq[2][4];
#pragma unroll
  for (int nq = 0; nq < 2; ++nq)
#pragma unroll
    for (int j = 0; j < 4; ++j) dq[nq][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int tw0 = bs + w0;
  for (int it = 0; it <= qt0; ++it) {
    const int kt = bs + it * 64;
    const bf16* Kt = blk + (1 * NT + it) * 4096;
    const bf16* Vt = blk + (2 * NT + it) * 4096;
    bf16x8 kf[4][2], vf[4][2], ktf[4][2];
#pragma unroll
    for (int ku = 0; ku < 4; ++ku)
#pragma unroll
      for (int ds = 0; ds < 2; ++ds) {
        kf[ku][ds] = trow8a(Kt, ku * 16 + lr, ds * 32 + lg * 8);
        vf[ku][ds] = trow8a(Vt, ku * 16 + lr, ds * 32 + lg * 8);
      }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int us = 0; us < 2; ++us) ktf[j][us] = tcol8p(Kt, us * 32, j, lane);
    lds_tr_wait();
#pragma unroll
    for (int ku = 0; ku < 4; ++ku)
#pragma unroll
      for (int ds = 0; ds < 2; ++ds) {
        lds_tr_bind(kf[ku][ds]);
        lds_tr_bind(vf[ku][ds]);
      }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int us = 0; us < 2; ++us) lds_tr_bind(ktf[j][us]);
#pragma unroll
    for (int nq = 0; nq < 2; ++nq) {
      const int tq = tw0 + nq * 16;
      if (tq >= be || tq + 15 < kt) continue;  // wave-uniform
      if (kt + 63 <= tq && tq + 15 < be)        // every key precedes every query
        blk_dq_group<false>(kf, vf, ktf, qf[nq], df[nq], ls[nq], dl[nq], dq[nq], kt, tq, be, sl2,
                            lane);
      else
        blk_dq_group<true>(kf, vf, ktf, qf[nq], df[nq], ls[nq], dl[nq], dq[nq], kt, tq, be, sl2,
                           lane);
    }
  }
#pragma unroll
  for (int nq = 0; nq < 2; ++nq) {
    const int t = tw0 + nq * 16 + lr;
    if (t < be) {
      bf16* pp = dst + (int64_t)t * rs + lg * 4;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        store4(pp + j * 16, dq[nq][j][0] * scale, dq[nq][j][1] * scale, dq[nq][j][2] * scale,
               dq[nq][j][3] * scale);
    }
  }
}

// Fused backward of one block for blocks of at most NW * 32 tokens:
// workgroup = (block, batch * head).  Q, K, V and dO of the whole block are
// loaded into LDS once (direct loads); each wave first forms delta_t =
// dO_t . O_t for its 32 queries, then owns 32 keys for dK and dV and finally
// its 32 queries for dQ.
template <int NW>
__global__ __launch_bounds__(NW * 64, NW >= 8 ? 1 : 2) void attn_bwd_block_bf16_kernel(
    const bf16* __restrict__ qkv, const bf16* __restrict__ o, const bf16* __restrict__ dout,
    const float* __restrict__ lse, bf16* __restrict__ dqkv, int Tn, int D, int H, int L,
    float sl2, float scale) {
  constexpr int NT = (NW * 32 + 63) / 64;  // 64-row tiles per matrix
  __shared__ __attribute__((aligned(1024))) bf16 lds[4][NT][64 * 64];  // Q, K, V, dO
  __shared__ __attribute__((aligned(16))) float ls_s[NT * 64], dl_s[NT * 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int b = blockIdx.z / H, h = blockIdx.z % H;
  const int bs = blockIdx.y * L;
  const int be = min(bs + L, Tn);
  const int ntile = (be - bs + 63) / 64;
  const int64_t rs = 3LL * D;
  const bf16* base = qkv + (int64_t)b * Tn * rs + h * kDh;
  const bf16* ob = o + (int64_t)b * Tn * D + h * kDh;
  const bf16* db = dout + (int64_t)b * Tn * D + h * kDh;
  const int64_t lrow = ((int64_t)b * H + h) * Tn;
  const int w0 = wave * 32;  // this wave's 32 queries (dQ) and keys (dK, dV), block-relative

  for (int it = 0; it < ntile; ++it) {
    const int r0 = bs + it * 64;
    tile_issue<NW>(base, rs, r0, be - 1, lds[0][it], wave, lane);
    tile_issue<NW>(base + D, rs, r0, be - 1, lds[1][it], wave, lane);
    tile_issue<NW>(base + 2 * D, rs, r0, be - 1, lds[2][it], wave, lane);
    tile_issue<NW>(db, D, r0, be - 1, lds[3][it], wave, lane);
  }
  // delta and lse of this wave's queries, while the tiles land.
#pragma unroll
  for (int nq = 0; nq < 2; ++nq) {
    const int tl = w0 + nq * 16 + lr;
    const int t = bs + tl;
    const bool ok = t < be;
    float part = 0.f;
#pragma unroll
    for (int ds = 0; ds < 2; ++ds) {
      const bf16x8 dfv = ok ? *reinterpret_cast<const bf16x8*>(db + (int64_t)t * D + ds * 32 + lg * 8) : bf16x8{};
      const bf16x8 ofv = ok ? *reinterpret_cast<const bf16x8*>(ob + (int64_t)t * D + ds * 32 + lg * 8) : bf16x8{};
#pragma unroll
      for (int e = 0; e < 8; ++e) part += (float)dfv[e] * (float)ofv[e];
    }
    part += __shfl_xor(part, 16, 64);
    part += __shfl_xor(part, 32, 64);
    if (lg == 0 && tl < NT * 64) {
      dl_s[tl] = part;
      ls_s[tl] = ok ? lse[lrow + t] : 0.f;
    }
  }
  vm_wait<0>();
  __syncthreads();

  bf16* dst = dqkv + (int64_t)b * Tn * rs + h * kDh;
  if (bs + w0 < be)
    blk_dkdv<NT>(&lds[0][0][0], ls_s, dl_s, dst, rs, D, bs, be, w0, ntile, sl2, scale, lane);
  if (bs + w0 < be) blk_dq<NT>(&lds[0][0][0], ls_s, dl_s, dst, rs, bs, be, w0, sl2, scale, lane);
}


// Waves per attention workgroup (1, 2 or 4), each owning 32 queries or keys.
int attn_waves(int L, int T) {
  const int lb = L < T ? L : T;
  const int w = (lb + 31) / 32;
  return w <= 1 ? 1 : (w == 2 ? 2 : 4);
}

template <typename E>
hipError_t attn_fwd_t(const void* qkv, void* out, float* lse, int B, int T, int D, int H, int L,
                      hipStream_t s) {
  const int nw = attn_waves(L, T);
  const int lb = L < T ? L : T;
  const int nb = (T + L - 1) / L;
  dim3 grid((lb + nw * 32 - 1) / (nw * 32), nb, B * H);
  const float sl2 = 1.4426950408889634f / sqrtf((float)kDh);
  hipLaunchKernelGGL(attn_fwd_kernel<E>, grid, dim3(nw * 64), 0, s, (const E*)qkv, (E*)out, lse,
                     T, D, H, L, sl2);
  return hipGetLastError();
}

template <typename E>
hipError_t attn_bwd_dq_t(const void* qkv, const void* o, const void* dout, const float* lse,
                         float* delta, void* dqkv, int B, int T, int D, int H, int L,
                         hipStream_t s) {
  const int nw = attn_waves(L, T);
  const int lb = L < T ? L : T;
  const int nb = (T + L - 1) / L;
  dim3 grid((lb + nw * 32 - 1) / (nw * 32), nb, B * H);
  const float scale = 1.0f / sqrtf((float)kDh);
  const float sl2 = 1.4426950408889634f * scale;
  hipLaunchKernelGGL(attn_bwd_dq_kernel<E>, grid, dim3(nw * 64), 0, s, (const E*)qkv,
                     (const E*)o, (const E*)dout, lse, delta, (E*)dqkv, T, D, H, L, sl2, scale);
  return hipGetLastError();
}

template <typename E>
hipError_t attn_bwd_dkdv_t(const void* qkv, const void* dout, const float* lse,
                           const float* delta, void* dqkv, int B, int T, int D, int H, int L,
                           hipStream_t s) {
  const int nw = attn_waves(L, T);
  const int lb = L < T ? L : T;
  const int nb = (T + L - 1) / L;
  dim3 grid((lb + nw * 32 - 1) / (nw * 32), nb, B * H);
  const float scale = 1.0f / sqrtf((float)kDh);
  const float sl2 = 1.4426950408889634f * scale;
  hipLaunchKernelGGL(attn_bwd_dkdv_kernel<E>, grid, dim3(nw * 64), 0, s, (const E*)qkv,
                     (const E*)dout, lse, delta, (E*)dqkv, T, D, H, L, sl2, scale);
  return hipGetLastError();
}

}  // namespace

hipError_t attn_fwd(DType dt, const void* qkv, void* out, float* lse, int B, int T, int D, int H,
                    int L, hipStream_t s) {
  if (attn_small_heads(D, H)) return attn_small_fwd(dt, qkv, out, lse, B, T, D, H, L, s);
  if (dt == DType::BF16) {
    const int nw = attn_waves(L, T);
    const int lb = L < T ? L : T;
    dim3 grid((lb + nw * 32 - 1) / (nw * 32), (T + L - 1) / L, B * H);
    const float sl2 = 1.4426950408889634f / sqrtf((float)kDh);
#define FWD(NW) hipLaunchKernelGGL(attn_fwd_bf16_kernel<NW>, grid, dim3(NW * 64), 0, s, (const bf16*)qkv, (bf16*)out, lse, T, D, H, L, sl2)
    if (nw == 1) FWD(1); else if (nw == 2) FWD(2); else FWD(4);
#undef FWD
    return hipGetLastError();
  }
  return attn_fwd_t<float>(qkv, out, lse, B, T, D, H, L, s);
}

hipError_t attn_bwd_dq(DType dt, const void* qkv, const void* out, const void* dout,
                       const float* lse, float* delta, void* dqkv, int B, int T, int D, int H,
                       int L, hipStream_t s) {
  if (attn_small_heads(D, H))
    return attn_small_dq(dt, qkv, out, dout, lse, delta, dqkv, B, T, D, H, L, s);
  if (dt == DType::BF16) {
    const int nw = attn_waves(L, T);
    const int lb = L < T ? L : T;
    dim3 grid((lb + nw * 32 - 1) / (nw * 32), (T + L - 1) / L, B * H);
    const float scale = 1.0f / sqrtf((float)kDh);
    const float sl2 = 1.4426950408889634f * scale;
#define DQ(NW) hipLaunchKernelGGL(attn_bwd_dq_bf16_kernel<NW>, grid, dim3(NW * 64), 0, s, (const bf16*)qkv, (const bf16*)out, (const bf16*)dout, lse, delta, (bf16*)dqkv, T, D, H, L, sl2, scale)
    if (nw == 1) DQ(1); else if (nw == 2) DQ(2); else DQ(4);
#undef DQ
    return hipGetLastError();
  }
  return attn_bwd_dq_t<float>(qkv, out, dout, lse, delta, dqkv, B, T, D, H, L, s);
}

bool attn_bwd_fused(DType dt, int T, int D, int H, int L) {
  const int lb = L < T ? L : T;
  return dt == DType::BF16 && lb <= 256 && !attn_small_heads(D, H);
}

hipError_t attn_bwd_block(DType dt, const void* qkv, const void* out, const void* dout,
                          const float* lse, void* dqkv, int B, int T, int D, int H, int L,
                          hipStream_t s) {
  if (!attn_bwd_fused(dt, T, D, H, L)) return hipErrorInvalidValue;
  const int lb = L < T ? L : T;
  const int nblk = (T + L - 1) / L;
  const float scale = 1.0f / sqrtf((float)kDh);
  const float sl2 = 1.4426950408889634f * scale;
  const int nw = lb <= 128 ? attn_waves(L, T) : 8;  // one wave per 32 tokens of the block
  dim3 grid(1, nblk, B * H);
#define BLK(NW) hipLaunchKernelGGL(attn_bwd_block_bf16_kernel<NW>, grid, dim3(NW * 64), 0, s, (const bf16*)qkv, (const bf16*)out, (const bf16*)dout, lse, (bf16*)dqkv, T, D, H, L, sl2, scale)
  if (nw == 1) BLK(1); else if (nw == 2) BLK(2); else if (nw == 4) BLK(4); else BLK(8);
#undef BLK
  return hipGetLastError();
}

hipError_t attn_bwd_dkdv(DType dt, const void* qkv, const void* dout, const float* lse,
                         const float* delta, void* dqkv, int B, int T, int D, int H, int L,
                         hipStream_t s) {
  if (attn_small_heads(D, H))
    return attn_small_dkdv(dt, qkv, dout, lse, delta, dqkv, B, T, D, H, L, s);
  if (dt == DType::BF16) {
    const int nw = attn_waves(L, T);
    const int lb = L < T ? L : T;
    dim3 grid((lb + nw * 32 - 1) / (nw * 32), (T + L - 1) / L, B * H);
    const float scale = 1.0f / sqrtf((float)kDh);
    const float sl2 = 1.4426950408889634f * scale;
#define DKDV(NW) hipLaunchKernelGGL(attn_bwd_dkdv_bf16_kernel<NW>, grid, dim3(NW * 64), 0, s, (const bf16*)qkv, (const bf16*)dout, lse, (const float*)delta, (bf16*)dqkv, T, D, H, L, sl2, scale)
    if (nw == 1) DKDV(1); else if (nw == 2) DKDV(2); else DKDV(4);
#undef DKDV
    return hipGetLastError();
  }
  return attn_bwd_dkdv_t<float>(qkv, dout, lse, delta, dqkv, B, T, D, H, L, s);
}

}  // namespace bcmt
