// Block-local causal attention (Sec. 3.3, 3.6) for heads of 16 or 32
// dimensions, the head width of the paper's own model (d_model = 128, 8
// heads, Sec. 4).  Two implementations with one interface (that of the
// 64-dim two-pass path):
//   forward  out [B, T, D] at columns h*dh..; lse [B, H, T] (base 2, of the
//            scores scaled by log2(e) / sqrt(dh));
//   dq pass  dq into dqkv, delta [B, H, T] = dO . O per query;
//   dkdv     dk, dv into dqkv.
// qkv and dqkv are [B, T, 3D] with Q | K | V, head h at columns h*dh.
//  - float32: plain vector arithmetic, one thread per query (per key in the
//    dK / dV pass), the other operand's rows staged through LDS in chunks
//    of kSmChunk tokens and read by broadcast, softmax in base 2 with a
//    running maximum;
//  - bf16: the matrix cores, with the tiling of the 64-dim kernels (32
//    queries or keys per wave, tiles of 64 tokens; a 16-wide head fills
//    half of the instruction's 32-deep step).
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

// ------------------------------------------------------------------ bf16 forward on the matrix cores
// The same flow as the 64-dimensional forward: per wave 32 queries (two
// groups of 16), keys in tiles of 64 staged with direct global->LDS loads
// (double buffered), scores and P V on v_mfma_f32_16x16x32_bf16.  A head of
// 32 dimensions is exactly one 32-deep step of the matrix instruction; a
// head of 16 is that step with the upper 16 dimensions zero (lane groups 2
// and 3 hold zeros for Q and K).  Tiles are [64 tokens][DH] with 16-byte
// chunks XOR-swizzled by row pairs; V^T operands come from the V tile
// through ds_read_b64_tr_b16.
template <int DH>
__device__ __forceinline__ int stoff(int r, int c) {
  constexpr int CM = DH / 8 - 1;  // chunk mask
  return r * DH + (((c >> 3) ^ ((r >> 1) & CM)) << 3) + (c & 7);
}
template <int DH>
__device__ __forceinline__ bf16x4 scol4(const bf16* t, int k0, int c0, int lane) {
  const int i = lane & 15;
  return lds_read_tr(t + stoff<DH>(k0 + (i >> 2), c0 + ((i & 3) << 2)));
}
// V^T operand over dims dsub*16 + lane%16 and the 32 keys
// {b0 + 4g .. +3} u {b0 + 16 + 4g .. +3} of lane group g.
template <int DH>
__device__ __forceinline__ bf16x8 scol8p(const bf16* t, int b0, int dsub, int lane) {
  const int g = lane >> 4;
  const bf16x4 a = scol4<DH>(t, b0 + 4 * g, dsub * 16, lane);
  const bf16x4 b = scol4<DH>(t, b0 + 16 + 4 * g, dsub * 16, lane);
  bf16x8 r = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  return r;
}

// This wave's share of the direct loads of two tiles (64 tokens from r0 of
// src0 and src1, row strides rs0 and rs1, rows clamped to rlast; clamped rows
// are never used unmasked).  Each load instruction moves 1 KB: 64 / (DH / 8)
// rows.
template <int NW, int DH>
__device__ __forceinline__ void pair_issue(const bf16* src0, int64_t rs0, const bf16* src1,
                                           int64_t rs1, int r0, int rlast, bf16* t0, bf16* t1,
                                           int wave, int lane) {
  constexpr int CPR = DH / 8;        // 16-byte chunks per row
  constexpr int PT = DH / 8;         // load instructions per tile
  constexpr int PW = 2 * PT / NW;    // per wave, both tiles together
  static_assert(PW >= 1 && (2 * PT) % NW == 0, "loads per wave");
#pragma unroll
  for (int i = 0; i < PW; ++i) {
    const int gi = wave * PW + i;
    const int tile = gi / PT, part = gi % PT;  // wave-uniform
    const int row = part * (64 / CPR) + lane / CPR;
    const int cg = (lane % CPR) ^ ((row >> 1) & (CPR - 1));
    const int grow = min(r0 + row, rlast);
    const bf16* src = tile == 0 ? src0 + (int64_t)grow * rs0 : src1 + (int64_t)grow * rs1;
    bf16* dst = (tile == 0 ? t0 : t1) + part * 512;
    __builtin_amdgcn_global_load_lds(src + cg * 8, (lds_void_t*)dst, 16, 0, 0);
  }
}
// 64 floats (one per lane), indices clamped to last.
__device__ __forceinline__ void vec64_issue(const float* src, int i0, int last, float* dst,
                                            int lane) {
  __builtin_amdgcn_global_load_lds(src + min(i0 + lane, last), (lds_void_t*)dst, 4, 0, 0);
}
// Row fragment (8 dimensions from lg * 8) of tile row r; zero past the head.
template <int DH>
__device__ __forceinline__ bf16x8 srow8(const bf16* t, int r, int lg) {
  return lg * 8 < DH ? *reinterpret_cast<const bf16x8*>(t + stoff<DH>(r, lg * 8)) : bf16x8{};
}
// The same from global memory (row pointer p).
template <int DH>
__device__ __forceinline__ bf16x8 grow8(const bf16* p, bool ok, int lg) {
  return ok && lg * 8 < DH ? *reinterpret_cast<const bf16x8*>(p + lg * 8) : bf16x8{};
}

template <int N>
__device__ __forceinline__ void sm_vm_wait() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

template <int NW, int DH>
__global__ __launch_bounds__(NW * 64) void attn_small_fwd_mfma_kernel(
    const bf16* __restrict__ qkv, bf16* __restrict__ out, float* __restrict__ lse, int Tn, int D,
    int H, int L, float sl2) {
  constexpr int QT = NW * 32;
  constexpr int NI = 2 * (DH / 8) / NW;  // direct loads per wave per K / V tile pair
  constexpr int NJ = DH / 16;            // 16-wide column tiles of the output
  __shared__ __attribute__((aligned(1024))) bf16 lds[2][2][64 * DH];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int b = blockIdx.z / H, h = blockIdx.z % H;
  const int bs = blockIdx.y * L;
  const int be = min(bs + L, Tn);
  const int q0 = bs + blockIdx.x * QT;
  if (q0 >= be) return;
  const int64_t rs = 3LL * D;
  const bf16* base = qkv + (int64_t)b * Tn * rs + h * DH;
  const int tw0 = q0 + wave * 32;
  const int kend = min(be, q0 + QT);
  const int nt = (kend - bs + 63) / 64;

  bf16x8 qf[2];
#pragma unroll
  for (int nq = 0; nq < 2; ++nq) {
    const int t = tw0 + nq * 16 + lr;
    qf[nq] = grow8<DH>(base + (int64_t)t * rs, t < be, lg);
  }
  f32x4 o[2][NJ];
  float m[2], l[2];
#pragma unroll
  for (int nq = 0; nq < 2; ++nq) {
    m[nq] = -INFINITY;
    l[nq] = 0.f;
#pragma unroll
    for (int j = 0; j < NJ; ++j) o[nq][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  pair_issue<NW, DH>(base + D, rs, base + 2 * D, rs, bs, kend - 1, lds[0][0], lds[0][1], wave,
                    lane);
  if (nt > 1)
    pair_issue<NW, DH>(base + D, rs, base + 2 * D, rs, bs + 64, kend - 1, lds[1][0], lds[1][1],
                      wave, lane);
  for (int it = 0; it < nt; ++it) {
    if (it + 1 < nt) sm_vm_wait<NI>();
    else sm_vm_wait<0>();
    __builtin_amdgcn_s_barrier();
    const int kt = bs + it * 64;
    const bf16* Kt = lds[it & 1][0];
    const bf16* Vt = lds[it & 1][1];
    bool live[2];
#pragma unroll
    for (int nq = 0; nq < 2; ++nq) {
      const int tq = tw0 + nq * 16;
      live[nq] = !(tq >= be || tq + 15 < kt);  // wave-uniform
    }
    f32x4 s[2][4];
    if (live[0] || live[1]) {
      bf16x8 kf[4];
#pragma unroll
      for (int ku = 0; ku < 4; ++ku) kf[ku] = srow8<DH>(Kt, ku * 16 + lr, lg);
#pragma unroll
      for (int nq = 0; nq < 2; ++nq)
#pragma unroll
        for (int ku = 0; ku < 4; ++ku) s[nq][ku] = mma16(kf[ku], qf[nq], f32x4{0.f, 0.f, 0.f, 0.f});
    }
#pragma unroll
    for (int nq = 0; nq < 2; ++nq) {
      if (!live[nq]) continue;
      const int tq = tw0 + nq * 16;
      const int t_eff = min(tq + lr, be - 1);
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
      for (int j = 0; j < NJ; ++j) o[nq][j] *= alpha;
    }
    if (live[0] || live[1]) {
      bf16x8 vf[NJ][2];
#pragma unroll
      for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int us = 0; us < 2; ++us) vf[j][us] = scol8p<DH>(Vt, us * 32, j, lane);
      lds_tr_wait();
#pragma unroll
      for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int us = 0; us < 2; ++us) lds_tr_bind(vf[j][us]);
#pragma unroll
      for (int nq = 0; nq < 2; ++nq) {
        if (!live[nq]) continue;
#pragma unroll
        for (int us = 0; us < 2; ++us) {
          const bf16x8 pf = frag_from<bf16>(s[nq][2 * us], s[nq][2 * us + 1]);
#pragma unroll
          for (int j = 0; j < NJ; ++j) o[nq][j] = mma16(vf[j][us], pf, o[nq][j]);
        }
      }
    }
    if (it + 2 < nt) {
      __builtin_amdgcn_s_barrier();  // every wave is done with this buffer
      pair_issue<NW, DH>(base + D, rs, base + 2 * D, rs, kt + 128, kend - 1, lds[it & 1][0],
                        lds[it & 1][1], wave, lane);
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
      bf16* op = out + ((int64_t)b * Tn + t) * D + h * DH + lg * 4;
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        store4(op + j * 16, o[nq][j][0] * inv, o[nq][j][1] * inv, o[nq][j][2] * inv,
               o[nq][j][3] * inv);
      if (lg == 0) lse[((int64_t)b * H + h) * Tn + t] = m[nq] + log2f(lt);
    }
  }
}

// dQ on the matrix cores (same tiling as the forward): per key tile,
// scores S = K Q^T and dP = V dO^T, dS = P (dP - delta) with
// P = 2^(S sl2 - lse), then dQ += K^T dS.  Writes delta_t = dO_t . O_t,
// which the dK / dV pass reads.
template <int NW, int DH>
__global__ __launch_bounds__(NW * 64) void attn_small_dq_mfma_kernel(
    const bf16* __restrict__ qkv, const bf16* __restrict__ o, const bf16* __restrict__ dout,
    const float* __restrict__ lse, float* __restrict__ delta, bf16* __restrict__ dqkv, int Tn,
    int D, int H, int L, float sl2, float scale) {
  constexpr int QT = NW * 32;
  constexpr int NI = 2 * (DH / 8) / NW;
  constexpr int NJ = DH / 16;
  __shared__ __attribute__((aligned(1024))) bf16 lds[2][2][64 * DH];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int b = blockIdx.z / H, h = blockIdx.z % H;
  const int bs = blockIdx.y * L;
  const int be = min(bs + L, Tn);
  const int q0 = bs + blockIdx.x * QT;
  if (q0 >= be) return;
  const int64_t rs = 3LL * D;
  const bf16* base = qkv + (int64_t)b * Tn * rs + h * DH;
  const bf16* ob = o + (int64_t)b * Tn * D + h * DH;
  const bf16* db = dout + (int64_t)b * Tn * D + h * DH;
  const int64_t lrow = ((int64_t)b * H + h) * Tn;
  const int tw0 = q0 + wave * 32;
  const int kend = min(be, q0 + QT);
  const int nt = (kend - bs + 63) / 64;

  bf16x8 qf[2], df[2];
  float dl[2], ls[2];
#pragma unroll
  for (int nq = 0; nq < 2; ++nq) {
    const int t = tw0 + nq * 16 + lr;
    const bool ok = t < be;
    qf[nq] = grow8<DH>(base + (int64_t)t * rs, ok, lg);
    df[nq] = grow8<DH>(db + (int64_t)t * D, ok, lg);
    const bf16x8 of = grow8<DH>(ob + (int64_t)t * D, ok, lg);
    float part = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) part += (float)df[nq][e] * (float)of[e];
    part += __shfl_xor(part, 16, 64);
    part += __shfl_xor(part, 32, 64);
    dl[nq] = part;
    ls[nq] = ok ? lse[lrow + t] : 0.f;
    if (ok && lg == 0) delta[lrow + t] = part;
  }
  f32x4 dq[2][NJ];
#pragma unroll
  for (int nq = 0; nq < 2; ++nq)
#pragma unroll
    for (int j = 0; j < NJ; ++j) dq[nq][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  pair_issue<NW, DH>(base + D, rs, base + 2 * D, rs, bs, kend - 1, lds[0][0], lds[0][1], wave,
                    lane);
  if (nt > 1)
    pair_issue<NW, DH>(base + D, rs, base + 2 * D, rs, bs + 64, kend - 1, lds[1][0], lds[1][1],
                      wave, lane);
  for (int it = 0; it < nt; ++it) {
    if (it + 1 < nt) sm_vm_wait<NI>();
    else sm_vm_wait<0>();
    __builtin_amdgcn_s_barrier();
    const int kt = bs + it * 64;
    const bf16* Kt = lds[it & 1][0];
    const bf16* Vt = lds[it & 1][1];
    bf16x8 kf[4], vf[4], ktf[NJ][2];
#pragma unroll
    for (int ku = 0; ku < 4; ++ku) {
      kf[ku] = srow8<DH>(Kt, ku * 16 + lr, lg);
      vf[ku] = srow8<DH>(Vt, ku * 16 + lr, lg);
    }
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int us = 0; us < 2; ++us) ktf[j][us] = scol8p<DH>(Kt, us * 32, j, lane);
    lds_tr_wait();
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int us = 0; us < 2; ++us) lds_tr_bind(ktf[j][us]);
#pragma unroll
    for (int nq = 0; nq < 2; ++nq) {
      const int tq = tw0 + nq * 16;
      if (tq >= be || tq + 15 < kt) continue;  // wave-uniform
      f32x4 sc[4];
#pragma unroll
      for (int ku = 0; ku < 4; ++ku) {
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};
        const f32x4 sv = mma16(kf[ku], qf[nq], z);
        const f32x4 dp = mma16(vf[ku], df[nq], z);
        const int t_eff = min(tq + lr, be - 1);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int u = kt + ku * 16 + lg * 4 + r;
          const float pv = u <= t_eff ? exp2_fast(sv[r] * sl2 - ls[nq]) : 0.f;
          sc[ku][r] = pv * (dp[r] - dl[nq]);
        }
      }
#pragma unroll
      for (int us = 0; us < 2; ++us) {
        const bf16x8 zf = frag_from<bf16>(sc[2 * us], sc[2 * us + 1]);
#pragma unroll
        for (int j = 0; j < NJ; ++j) dq[nq][j] = mma16(ktf[j][us], zf, dq[nq][j]);
      }
    }
    if (it + 2 < nt) {
      __builtin_amdgcn_s_barrier();
      pair_issue<NW, DH>(base + D, rs, base + 2 * D, rs, kt + 128, kend - 1, lds[it & 1][0],
                        lds[it & 1][1], wave, lane);
    }
  }

#pragma unroll
  for (int nq = 0; nq < 2; ++nq) {
    const int t = tw0 + nq * 16 + lr;
    if (t < be) {
      bf16* p = dqkv + ((int64_t)b * Tn + t) * rs + h * DH + lg * 4;
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        store4(p + j * 16, dq[nq][j][0] * scale, dq[nq][j][1] * scale, dq[nq][j][2] * scale,
               dq[nq][j][3] * scale);
    }
  }
}

// dK / dV on the matrix cores: per wave 32 keys (two groups of 16); query
// tiles of 64 from the workgroup's first key on, with their lse and delta,
// staged by direct loads.  S = Q K^T and dP = dO V^T per tile; then
// dV += dO^T P and dK += Q^T dS.
template <int NW, int DH>
__global__ __launch_bounds__(NW * 64) void attn_small_dkdv_mfma_kernel(
    const bf16* __restrict__ qkv, const bf16* __restrict__ dout, const float* __restrict__ lse,
    const float* __restrict__ delta, bf16* __restrict__ dqkv, int Tn, int D, int H, int L,
    float sl2, float scale) {
  constexpr int KT = NW * 32;
  constexpr int NI = 2 * (DH / 8) / NW;
  constexpr int NJ = DH / 16;
  __shared__ __attribute__((aligned(1024))) bf16 lds[2][2][64 * DH];
  __shared__ __attribute__((aligned(16))) float vec_s[2][2][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int b = blockIdx.z / H, h = blockIdx.z % H;
  const int bs = blockIdx.y * L;
  const int be = min(bs + L, Tn);
  const int k0 = bs + blockIdx.x * KT;
  if (k0 >= be) return;
  const int64_t rs = 3LL * D;
  const bf16* base = qkv + (int64_t)b * Tn * rs + h * DH;
  const bf16* db = dout + (int64_t)b * Tn * D + h * DH;
  const int64_t lrow = ((int64_t)b * H + h) * Tn;
  const int uw0 = k0 + wave * 32;
  const int nt = (be - k0 + 63) / 64;

  bf16x8 kf[2], vf[2];
#pragma unroll
  for (int ku = 0; ku < 2; ++ku) {
    const int u = uw0 + ku * 16 + lr;
    kf[ku] = grow8<DH>(base + D + (int64_t)u * rs, u < be, lg);
    vf[ku] = grow8<DH>(base + 2 * D + (int64_t)u * rs, u < be, lg);
  }
  f32x4 dk[2][NJ], dv[2][NJ];
#pragma unroll
  for (int ku = 0; ku < 2; ++ku)
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      dk[ku][j] = f32x4{0.f, 0.f, 0.f, 0.f};
      dv[ku][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

  auto issue = [&](int tt, int buf) {
    pair_issue<NW, DH>(base, rs, db, D, tt, be - 1, lds[buf][0], lds[buf][1], wave, lane);
    if (wave == 0) {
      vec64_issue(lse + lrow, tt, be - 1, vec_s[buf][0], lane);
      vec64_issue(delta + lrow, tt, be - 1, vec_s[buf][1], lane);
    }
  };
  issue(k0, 0);
  if (nt > 1) issue(k0 + 64, 1);
  for (int it = 0; it < nt; ++it) {
    if (it + 1 < nt) {
      if (wave == 0) sm_vm_wait<NI + 2>();
      else sm_vm_wait<NI>();
    } else {
      sm_vm_wait<0>();
    }
    __builtin_amdgcn_s_barrier();
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
        const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
        const f32x4 sv = mma16(srow8<DH>(Qt, ts * 16 + lr, lg), kf[ku], zero);
        const f32x4 dp = mma16(srow8<DH>(Dt, ts * 16 + lr, lg), vf[ku], zero);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = tt + ts * 16 + lg * 4 + r;
          const bool ok = t >= u && t < be && u < be;
          const float pv = ok ? exp2_fast(sv[r] * sl2 - lsv[ts][r]) : 0.f;
          p[ts][r] = pv;
          z[ts][r] = pv * (dp[r] - dlv[ts][r]);
        }
      }
#pragma unroll
      for (int tq = 0; tq < 2; ++tq) {
        const bf16x8 pf = frag_from<bf16>(p[2 * tq], p[2 * tq + 1]);
        const bf16x8 zf = frag_from<bf16>(z[2 * tq], z[2 * tq + 1]);
        bf16x8 dtf[NJ], qtf[NJ];
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          dtf[j] = scol8p<DH>(Dt, tq * 32, j, lane);
          qtf[j] = scol8p<DH>(Qt, tq * 32, j, lane);
        }
        lds_tr_wait();
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          lds_tr_bind(dtf[j]);
          lds_tr_bind(qtf[j]);
        }
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          dv[ku][j] = mma16(dtf[j], pf, dv[ku][j]);
          dk[ku][j] = mma16(qtf[j], zf, dk[ku][j]);
        }
      }
    }
    if (it + 2 < nt) {
      __builtin_amdgcn_s_barrier();
      issue(tt + 128, it & 1);
    }
  }

#pragma unroll
  for (int ku = 0; ku < 2; ++ku) {
    const int u = uw0 + ku * 16 + lr;
    if (u < be) {
      bf16* p = dqkv + ((int64_t)b * Tn + u) * rs + h * DH + lg * 4;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        store4(p + D + j * 16, dk[ku][j][0] * scale, dk[ku][j][1] * scale, dk[ku][j][2] * scale,
               dk[ku][j][3] * scale);
        store4(p + 2 * D + j * 16, dv[ku][j][0], dv[ku][j][1], dv[ku][j][2], dv[ku][j][3]);
      }
    }
  }
}

// Waves per matrix-core workgroup (each owns 32 queries or keys).
int small_waves(int lb) { return lb <= 32 ? 1 : (lb <= 64 ? 2 : 4); }

template <int DH>
hipError_t small_bwd_mfma(int pass, const void* qkv, const void* o, const void* dout,
                          const float* lse, float* delta, void* dqkv, int B, int Tn, int D, int H,
                          int L, hipStream_t s) {
  const int lb = L < Tn ? L : Tn;
  const int nw = small_waves(lb);
  const dim3 grid((lb + nw * 32 - 1) / (nw * 32), (Tn + L - 1) / L, B * H);
  const float scale = 1.0f / sqrtf((float)DH);
  const float sl2 = 1.4426950408889634f * scale;
#define SDQ(NW)                                                                               \
  hipLaunchKernelGGL((attn_small_dq_mfma_kernel<NW, DH>), grid, dim3(NW * 64), 0, s,           \
                     (const bf16*)qkv, (const bf16*)o, (const bf16*)dout, lse, delta,           \
                     (bf16*)dqkv, Tn, D, H, L, sl2, scale)
#define SDKDV(NW)                                                                             \
  hipLaunchKernelGGL((attn_small_dkdv_mfma_kernel<NW, DH>), grid, dim3(NW * 64), 0, s,         \
                     (const bf16*)qkv, (const bf16*)dout, lse, (const float*)delta,             \
                     (bf16*)dqkv, Tn, D, H, L, sl2, scale)
  if (pass == 1) {
    if (nw == 1) SDQ(1);
    else if (nw == 2) SDQ(2);
    else SDQ(4);
  } else {
    if (nw == 1) SDKDV(1);
    else if (nw == 2) SDKDV(2);
    else SDKDV(4);
  }
#undef SDQ
#undef SDKDV
  return hipGetLastError();
}

template <int DH>
hipError_t small_fwd_mfma(const void* qkv, void* out, float* lse, int B, int Tn, int D, int H,
                          int L, hipStream_t s) {
  const int lb = L < Tn ? L : Tn;
  const int nw = small_waves(lb);
  const dim3 grid((lb + nw * 32 - 1) / (nw * 32), (Tn + L - 1) / L, B * H);
  const float sl2 = 1.4426950408889634f / sqrtf((float)DH);
#define SFWD(NW)                                                                              \
  hipLaunchKernelGGL((attn_small_fwd_mfma_kernel<NW, DH>), grid, dim3(NW * 64), 0, s,          \
                     (const bf16*)qkv, (bf16*)out, lse, Tn, D, H, L, sl2)
  if (nw == 1) SFWD(1);
  else if (nw == 2) SFWD(2);
  else SFWD(4);
#undef SFWD
  return hipGetLastError();
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
  if (dt == DType::BF16) {  // the matrix cores
    if (D / H == 16) return small_fwd_mfma<16>(qkv, out, lse, B, T, D, H, L, s);
    if (D / H == 32) return small_fwd_mfma<32>(qkv, out, lse, B, T, D, H, L, s);
    return hipErrorInvalidValue;
  }
  return small_dispatch<float>(0, qkv, nullptr, nullptr, out, lse, nullptr, B, T, D, H, L, s);
}

hipError_t attn_small_dq(DType dt, const void* qkv, const void* o, const void* dout,
                         const float* lse, float* delta, void* dqkv, int B, int T, int D, int H,
                         int L, hipStream_t s) {
  if (dt == DType::BF16) {  // the matrix cores
    if (D / H == 16) return small_bwd_mfma<16>(1, qkv, o, dout, lse, delta, dqkv, B, T, D, H, L, s);
    if (D / H == 32) return small_bwd_mfma<32>(1, qkv, o, dout, lse, delta, dqkv, B, T, D, H, L, s);
    return hipErrorInvalidValue;
  }
  return small_dispatch<float>(1, qkv, o, dout, dqkv, const_cast<float*>(lse), delta, B, T, D, H,
                               L, s);
}

hipError_t attn_small_dkdv(DType dt, const void* qkv, const void* dout, const float* lse,
                           const float* delta, void* dqkv, int B, int T, int D, int H, int L,
                           hipStream_t s) {
  if (dt == DType::BF16) {
    if (D / H == 16)
      return small_bwd_mfma<16>(2, qkv, nullptr, dout, lse, const_cast<float*>(delta), dqkv, B, T,
                                D, H, L, s);
    if (D / H == 32)
      return small_bwd_mfma<32>(2, qkv, nullptr, dout, lse, const_cast<float*>(delta), dqkv, B, T,
                                D, H, L, s);
    return hipErrorInvalidValue;
  }
  return small_dispatch<float>(2, qkv, nullptr, dout, dqkv, const_cast<float*>(lse),
                               const_cast<float*>(delta), B, T, D, H, L, s);
}

}  // namespace bcmt
