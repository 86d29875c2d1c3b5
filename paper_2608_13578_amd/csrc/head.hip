// The tied output head of the language model (Sec. 4.1: logits z = f E^T
// over the vocabulary, mean cross-entropy) without stored logits, for a
// feature width of 128.
//
// A workgroup takes 128 rows of f (four waves of 32, kept in registers as
// matrix-instruction operands for the whole kernel) and one contiguous
// range of the vocabulary, which it streams through LDS in tiles of 64
// rows of E (16 KB, a ring of three, filled by direct global->LDS loads).
// Per tile each wave forms its 32 x 64 logits on the matrix cores and
// consumes them in registers:
//   statistics pass: a running max and sum of exp(z - max) per row (online
//     softmax, base 2), one (max, sum) pair per row and vocabulary range at
//     the end, which the log-sum-exp kernel combines;
//   gradient pass: g = (softmax(z) - onehot(target)) / n from the row's
//     log-sum-exp, stored as bf16 for the product dE = G^T f, and df = G E
//     accumulated on the matrix cores from the same E tile (read
//     transposed) and the g values held in registers; one float32 partial
//     of df per vocabulary range, added in a fixed order afterwards.
// So the logits never reach memory, the per-tile pipeline fill and the
// statistics epilogue of a tiled product are gone, and df needs no pass
// over G.  The vocabulary ranges (grid x) give the launch several hundred
// workgroups at any number of rows; consecutive workgroups take different
// ranges, so each XCD's L2 serves one range of E to all row blocks.
#include "common.h"
#include "kernels.h"

namespace bcmt {
namespace {

constexpr int kHd = 128;      // feature width of this path
constexpr int kHRows = 128;   // rows of f per workgroup
constexpr int kHVt = 64;      // vocabulary rows per LDS tile
constexpr int kHThreads = 256;
constexpr int kHRing = 3;     // LDS tiles in flight
constexpr int kHLoads = kHVt * kHd * 2 / 1024 / 4;  // 1 KB direct loads per wave per tile
constexpr float kHL2e = 1.4426950408889634f;
constexpr float kHNone = -1e30f;  // running max before any valid column

// E tile in LDS: [64 rows][128] bf16, 256-byte rows; the 16-byte chunk c of
// row r sits at chunk c ^ eswz(r).  The logits instruction for vocabulary
// group ku reads, on lane i, row vrow(ku, i) = 16 (i / 4) + 4 ku + i % 4, so
// that lane group g ends up with 16 consecutive columns 16 g .. 16 g + 15 of
// the tile (four groups ku of four); its 16 rows differ in bits 0-1 and 4-5,
// which eswz maps one to one onto the four chunk bits.  A transposing read
// (16 lanes: two adjacent chunks of rows 16 g + 8 us + 4 h + 0..3) needs
// those four rows on disjoint chunk pairs: row bits 0-1 go to chunk bits
// 1-2; the next lane group (row bit 4) moves to the other half through
// chunk bit 3.
__device__ __forceinline__ int eswz(int r) {
  return ((r & 3) << 1) | (((r >> 4) & 1) << 3) | ((r >> 5) & 1);
}
__device__ __forceinline__ int eoff(int r, int c) {
  return r * kHd + (((c >> 3) ^ eswz(r)) << 3) + (c & 7);
}
__device__ __forceinline__ int vrow(int ku, int i) { return 16 * (i >> 2) + 4 * ku + (i & 3); }

// This wave's direct loads of vocabulary rows v0 .. v0+63 of E into tile t.
// Load i covers rows 4i .. 4i+3; lane l lands at chunk l % 16 of row
// 4i + l / 16 and so fetches global chunk (l % 16) ^ eswz(row).
__device__ __forceinline__ void etile_issue(const bf16* E, int v0, bf16* t, int wave, int lane) {
#pragma unroll
  for (int i = 0; i < kHLoads; ++i) {
    const int gi = wave * kHLoads + i;
    const int row = gi * 4 + (lane >> 4);
    const int cg = (lane & 15) ^ eswz(row);
    __builtin_amdgcn_global_load_lds(E + (int64_t)(v0 + row) * kHd + cg * 8,
                                     (lds_void_t*)(t + gi * 512), 16, 0, 0);
  }
}

template <int N>
__device__ __forceinline__ void hvm_wait() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Operand over the features 16 j + lane % 16 and, on lane group g, the
// vocabulary rows 16 g + 8 us + 0..7: the eight columns lane group g of a
// logits tile holds as its K-step us.
__device__ __forceinline__ bf16x8 ecol8(const bf16* t, int us, int j, int lane) {
  const int i = lane & 15, g = lane >> 4;
  const int c = j * 16 + ((i & 3) << 2);
  const int r = 16 * g + 8 * us + (i >> 2);
  const bf16x4 a = lds_read_tr(t + eoff(r, c));
  const bf16x4 b = lds_read_tr(t + eoff(r + 4, c));
  bf16x8 o = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  return o;
}

// GRAD false: part[2 (row nrange + range)] = (max z, sum exp(z - max)) over
// the range's columns below V (natural units; a range without such columns
// gives (-1e30, 0)).  GRAD true: G[row][v] for the range's columns
// (zero for v >= V) and dfp[range][row][0..127] = sum over the range of
// g[row][v] E[v][:].  Rows at or beyond `rows` are computed on zeros and
// never stored.
template <bool GRAD>
__global__ __launch_bounds__(kHThreads, 2) void head_kernel(
    const bf16* __restrict__ f, const bf16* __restrict__ E, int rows, int V, int ntiles, int tps,
    float* __restrict__ part, const float* __restrict__ lse, const int32_t* __restrict__ tgt,
    float inv_n, bf16* __restrict__ G, int64_t ldg, float* __restrict__ dfp) {
  __shared__ __attribute__((aligned(1024))) bf16 lds[kHRing][kHVt * kHd];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int range = blockIdx.x, nrange = gridDim.x;
  const int t0 = range * tps;
  const int nt = min(ntiles, t0 + tps) - t0;
  const int r0 = blockIdx.y * kHRows + wave * 32;

  // this wave's rows of f as the B operand of the logits (4 K steps of 32)
  bf16x8 qf[2][4];
  float lse2[2] = {0.f, 0.f};
  int tk[2] = {-1, -1};
#pragma unroll
  for (int nq = 0; nq < 2; ++nq) {
    const int row = r0 + nq * 16 + lr;
    const bool ok = row < rows;
#pragma unroll
    for (int ds = 0; ds < 4; ++ds)
      qf[nq][ds] = ok ? *reinterpret_cast<const bf16x8*>(f + (int64_t)row * kHd + ds * 32 + lg * 8)
                      : bf16x8{};
    if constexpr (GRAD) {
      const int rc = ok ? row : 0;
      lse2[nq] = lse[rc] * kHL2e - log2f(inv_n);  // exp2(z log2 e - lse2) = e^(z - lse) / n
      tk[nq] = min(max(tgt[rc], 0), V - 1);
    }
  }
  // statistics: a running max and sum per lane (its row, its 16 columns of
  // every tile), combined over the row's four lanes at the end
  float m[2] = {kHNone, kHNone}, l[2] = {0.f, 0.f};
  f32x4 o[2][8];
  if constexpr (GRAD) {
#pragma unroll
    for (int nq = 0; nq < 2; ++nq)
#pragma unroll
      for (int j = 0; j < 8; ++j) o[nq][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // Ring of three tiles: tile it + 2 is issued into the buffer tile it - 1
  // used, after the barrier that starts iteration it (every wave is past
  // its reads).  The only loads issued after tile it's are tile it + 1's,
  // so waiting until at most that many of this wave's memory operations are
  // outstanding means tile it has landed (loads complete in order); the
  // gradient pass's stores in between can only make the wait longer.
  if (nt > 0) etile_issue(E, t0 * kHVt, lds[0], wave, lane);
  if (nt > 1) etile_issue(E, (t0 + 1) * kHVt, lds[1], wave, lane);
  for (int it = 0; it < nt; ++it) {
    if (it + 1 < nt) hvm_wait<kHLoads>();
    else hvm_wait<0>();
    __builtin_amdgcn_s_barrier();
    if (it + 2 < nt) etile_issue(E, (t0 + it + 2) * kHVt, lds[(it + 2) % kHRing], wave, lane);
    const bf16* Et = lds[it % kHRing];
    const int v0 = (t0 + it) * kHVt;

    // logits: lane (lr, lg) holds row r0 + 16 nq + lr, columns
    // v0 + 16 lg + 4 ku + 0..3
    f32x4 s[2][4];
#pragma unroll
    for (int nq = 0; nq < 2; ++nq)
#pragma unroll
      for (int ku = 0; ku < 4; ++ku) s[nq][ku] = f32x4{0.f, 0.f, 0.f, 0.f};
    constexpr int KB = GRAD ? 2 : 4;  // vocabulary groups whose fragments are read at once
#pragma unroll
    for (int k0 = 0; k0 < 4; k0 += KB) {
      bf16x8 kf[KB][4];
#pragma unroll
      for (int u = 0; u < KB; ++u)
#pragma unroll
        for (int ds = 0; ds < 4; ++ds)
          kf[u][ds] = lds_read_b128(Et + eoff(vrow(k0 + u, lr), ds * 32 + lg * 8));
      lds_tr_wait();
#pragma unroll
      for (int u = 0; u < KB; ++u)
#pragma unroll
        for (int ds = 0; ds < 4; ++ds) lds_tr_bind(kf[u][ds]);
      // independent accumulators back to back
#pragma unroll
      for (int ds = 0; ds < 4; ++ds)
#pragma unroll
        for (int u = 0; u < KB; ++u)
#pragma unroll
          for (int nq = 0; nq < 2; ++nq)
            s[nq][k0 + u] = mma16(kf[u][ds], qf[nq][ds], s[nq][k0 + u]);
    }
    const int vb = v0 + 16 * lg;
    // Only the last tile of the vocabulary has columns at or beyond V: the
    // others skip the mask (wave-uniform).
    const bool masked = v0 + kHVt > V;
    if (masked) {
#pragma unroll
      for (int nq = 0; nq < 2; ++nq)
#pragma unroll
        for (int ku = 0; ku < 4; ++ku)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (vb + 4 * ku + r >= V) s[nq][ku][r] = -INFINITY;
    }

    if constexpr (!GRAD) {
      // m: running max of the raw logits; l: sum of exp(z - m), taken as
      // exp2(z log2 e - m log2 e) with the scaling folded into one fma
#pragma unroll
      for (int nq = 0; nq < 2; ++nq) {
        float mx = m[nq];
#pragma unroll
        for (int ku = 0; ku < 4; ++ku)
#pragma unroll
          for (int r = 0; r < 4; ++r) mx = fmaxf(mx, s[nq][ku][r]);
        const float c = mx * kHL2e;
        float ps = 0.f;
#pragma unroll
        for (int ku = 0; ku < 4; ++ku)
#pragma unroll
          for (int r = 0; r < 4; ++r) ps += exp2_fast(fmaf(s[nq][ku][r], kHL2e, -c));
        // (the difference first: m may be the -1e30 start value, whose
        // product with log2 e would not cancel exactly against c)
        l[nq] = fmaf(l[nq], exp2_fast((m[nq] - mx) * kHL2e), ps);
        m[nq] = mx;
      }
    } else {
      // g = exp(z - lse) / n - [v == target] / n, with 1/n folded into the
      // exponent; the target's correction only where a row's target falls
      // in this lane's 16 columns.  The bf16 values serve as G and as the
      // df instruction's B operand (K step us = columns 16 lg + 8 us + 0..7).
      bf16x8 pf[2][2];
#pragma unroll
      for (int nq = 0; nq < 2; ++nq) {
        float g[16];
#pragma unroll
        for (int ku = 0; ku < 4; ++ku)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            g[4 * ku + r] = exp2_fast(fmaf(s[nq][ku][r], kHL2e, -lse2[nq]));
        const int e = tk[nq] - vb;
        if (e >= 0 && e < 16) {
#pragma unroll
          for (int k = 0; k < 16; ++k)
            if (k == e) g[k] -= inv_n;
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          pf[nq][0][k] = (bf16)g[k];
          pf[nq][1][k] = (bf16)g[8 + k];
        }
        const int row = r0 + nq * 16 + lr;
        if (row < rows) {
          bf16* gp = G + (int64_t)row * ldg + vb;
          *reinterpret_cast<bf16x8*>(gp) = pf[nq][0];
          *reinterpret_cast<bf16x8*>(gp + 8) = pf[nq][1];
        }
      }
      // df += g E: A = E^T (feature rows, vocabulary in the logits' order),
      // B = g as stored; E^T fragments four at a time
#pragma unroll
      for (int us = 0; us < 2; ++us)
#pragma unroll
        for (int jh = 0; jh < 2; ++jh) {
          bf16x8 vf[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) vf[j] = ecol8(Et, us, 4 * jh + j, lane);
          lds_tr_wait();
#pragma unroll
          for (int j = 0; j < 4; ++j) lds_tr_bind(vf[j]);
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int nq = 0; nq < 2; ++nq)
              o[nq][4 * jh + j] = mma16(vf[j], pf[nq][us], o[nq][4 * jh + j]);
        }
    }
  }

  if constexpr (!GRAD) {
#pragma unroll
    for (int nq = 0; nq < 2; ++nq) {
      float mt = fmaxf(m[nq], __shfl_xor(m[nq], 16, 64));
      mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
      float lt = l[nq] * exp2_fast((m[nq] - mt) * kHL2e);
      lt += __shfl_xor(lt, 16, 64);
      lt += __shfl_xor(lt, 32, 64);
      const int row = r0 + nq * 16 + lr;
      if (lg == 0 && row < rows) {
        float* q = part + 2 * ((int64_t)row * nrange + range);
        q[0] = mt;
        q[1] = lt;
      }
    }
  } else {
    // lane holds row r0 + 16 nq + lr, features 16 j + 4 lg + 0..3
#pragma unroll
    for (int nq = 0; nq < 2; ++nq) {
      const int row = r0 + nq * 16 + lr;
      if (row >= rows) continue;
      float* dp = dfp + ((int64_t)range * rows + row) * kHd + lg * 4;
#pragma unroll
      for (int j = 0; j < 8; ++j) store4(dp + j * 16, o[nq][j][0], o[nq][j][1], o[nq][j][2], o[nq][j][3]);
    }
  }
}

struct HeadPlan {
  int rb, ntiles, tps, nrange;
};
// Vocabulary ranges: about `wgs` workgroups in all (two or three per CU,
// as registers allow), at most half as many ranges as 64-row tiles (so that
// the pairs fit the per-tile partial buffer of the tiled path), every
// range nonempty.
HeadPlan head_plan(int rows, int Vp, int wgs) {
  HeadPlan p;
  p.rb = (rows + kHRows - 1) / kHRows;
  p.ntiles = Vp / kHVt;
  int sp = wgs / p.rb;
  if (sp > p.ntiles / 2) sp = p.ntiles / 2;
  if (sp < 1) sp = 1;
  p.tps = (p.ntiles + sp - 1) / sp;
  p.nrange = (p.ntiles + p.tps - 1) / p.tps;
  return p;
}
constexpr int kStatsWgs = 768, kGradWgs = 512;

}  // namespace

bool head_fused_ok(int d, int Vp) { return d == kHd && Vp % 128 == 0 && Vp >= 128; }

size_t head_partial_bytes(int rows, int d, int Vp) {
  if (!head_fused_ok(d, Vp)) return 0;
  const HeadPlan p = head_plan(rows, Vp, kGradWgs);
  return (size_t)p.nrange * rows * kHd * sizeof(float);
}

hipError_t head_stats(const void* f, const void* E, int rows, int d, int V, int Vp, float* part,
                      int* nrange, hipStream_t s) {
  if (!head_fused_ok(d, Vp) || rows < 1 || V < 1 || V > Vp) return hipErrorInvalidValue;
  const HeadPlan p = head_plan(rows, Vp, kStatsWgs);
  *nrange = p.nrange;
  hipLaunchKernelGGL(head_kernel<false>, dim3(p.nrange, p.rb), dim3(kHThreads), 0, s,
                     (const bf16*)f, (const bf16*)E, rows, V, p.ntiles, p.tps, part,
                     (const float*)nullptr, (const int32_t*)nullptr, 0.f, (bf16*)nullptr,
                     (int64_t)0, (float*)nullptr);
  return hipGetLastError();
}

hipError_t head_grad(const void* f, const void* E, int rows, int d, int V, int Vp,
                     const float* lse, const int32_t* tgt, float inv_n, void* G, int64_t ldg,
                     float* dfpart, float* df, hipStream_t s) {
  if (!head_fused_ok(d, Vp) || rows < 1 || V < 1 || V > Vp) return hipErrorInvalidValue;
  const HeadPlan p = head_plan(rows, Vp, kGradWgs);
  float* out = p.nrange > 1 ? dfpart : df;
  hipLaunchKernelGGL(head_kernel<true>, dim3(p.nrange, p.rb), dim3(kHThreads), 0, s,
                     (const bf16*)f, (const bf16*)E, rows, V, p.ntiles, p.tps, (float*)nullptr,
                     lse, tgt, inv_n, (bf16*)G, ldg, out);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.nrange == 1) return e;
  return gemm_splitk_reduce(dfpart, p.nrange, rows, kHd, df, nullptr, nullptr, kHd, kHd, false, s);
}

}  // namespace bcmt
