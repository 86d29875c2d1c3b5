// A decoder-only language model built from BCMT layers: the architecture of
// the paper's experiments (Sec. 4.1: d_model, layers, heads, batch), with the
// parts the paper leaves unspecified read as a pre-LN decoder of its period:
//   x = E[tok] + Pe[t];
//   per layer: x += mix(LN1(x));  x += gelu(LN2(x) W1) W2   (hidden 4d)
//   logits = LNf(x) E^T (tied head);  loss = mean cross-entropy.
// mix is the BCMT layer (api.hip); with L >= T it is plain causal attention,
// the paper's Dense baseline.  Activations and the working copy of the
// parameters are bf16; the master parameters, their gradients and the AdamW
// moments are float32, in one flat vector each (layout: model_param_layout).
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>
#include <string.h>

#include <type_traits>

#include "../../include/bcmt.h"
#include "common.h"
#include "kernels.h"

namespace bcmt {
namespace {

constexpr float kLnEps = 1e-5f;
constexpr int kLnRowsPerGroup = 64;   // rows per workgroup of the LayerNorm backward
constexpr int kLnWaves = 16;          // waves per workgroup of the LayerNorm backward
constexpr int kWgradMinK = 128;     // split depth of the model's weight gradients
constexpr int kDfMinK = 512;        // split depth of the head's input gradient (K = vocabulary)

// ------------------------------------------------------------------ kernels

// x[r] = E[tok[r]] + Pe[r % T] for rows r = b T + t, 8 columns per thread.
// Token ids outside [0, V) are clamped (they are the caller's error).
__global__ __launch_bounds__(256) void embed_fwd_kernel(const int32_t* __restrict__ tok,
                                                        const bf16* __restrict__ E,
                                                        const bf16* __restrict__ Pe,
                                                        bf16* __restrict__ x, int rows, int T,
                                                        int d, int V) {
  const int per = d / 8;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)rows * per) return;
  const int r = (int)(i / per), c = (int)(i % per) * 8;
  const int tk = min(max(tok[r], 0), V - 1);
  float a[8], p[8];
  ld8(E + (int64_t)tk * d + c, a);
  ld8(Pe + (int64_t)(r % T) * d + c, p);
#pragma unroll
  for (int k = 0; k < 8; ++k) a[k] += p[k];
  st8(x + (int64_t)r * d + c, a);
}

// LayerNorm of x (+ y when given; the sum is rounded to bf16 and stored to
// xs, and normalised as rounded), one wave per row, d = 64 n (n <= 16).
__global__ __launch_bounds__(256) void add_ln_fwd_kernel(const bf16* __restrict__ x,
                                                         const bf16* __restrict__ y,
                                                         bf16* __restrict__ xs,
                                                         const float* __restrict__ g,
                                                         const float* __restrict__ b,
                                                         bf16* __restrict__ out,
                                                         float* __restrict__ mean,
                                                         float* __restrict__ rstd, int rows,
                                                         int d) {
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  const int n = d >> 6;
  const int64_t base = (int64_t)r * d + lane;
  float v[16];
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    if (j < n) {
      float a = (float)x[base + 64 * j];
      if (y) {
        const bf16 ab = (bf16)(a + (float)y[base + 64 * j]);
        xs[base + 64 * j] = ab;
        a = (float)ab;
      }
      v[j] = a;
      s += a;
    }
  }
  const float mu = wave_sum(s) / (float)d;
  float q = 0.f;
#pragma unroll
  for (int j = 0; j < 16; ++j)
    if (j < n) q += (v[j] - mu) * (v[j] - mu);
  const float rs = rsqrtf(wave_sum(q) / (float)d + kLnEps);
#pragma unroll
  for (int j = 0; j < 16; ++j)
    if (j < n) {
      const int c = lane + 64 * j;
      out[base + 64 * j] = (bf16)((v[j] - mu) * rs * g[c] + b[c]);
    }
  if (lane == 0) {
    mean[r] = mu;
    rstd[r] = rs;
  }
}

// LayerNorm backward: dx = dres + rstd (dxh - mean(dxh) - xh mean(dxh xh))
// with dxh = dy g (dres nullable; dx may alias dres), and this workgroup's
// partial sums of dy xh (gain) and dy (bias) over its rows into
// part[blockIdx.x][2][d].  Each of the 16 waves takes 4 consecutive rows,
// RB at a time with all their loads issued first; a lane holds up to NJ
// elements of a row (d <= 64 NJ).  Dynamic LDS: 16 * 2 * d floats.
template <typename TY, int NJ, int RB>
__global__ __launch_bounds__(1024) void ln_bwd_kernel(
    const TY* __restrict__ dy, const bf16* __restrict__ xs, const float* __restrict__ mean,
    const float* __restrict__ rstd, const float* __restrict__ g, const bf16* dres, bf16* dx,
    float* __restrict__ part, int rows, int d) {
  constexpr int RW = kLnRowsPerGroup / kLnWaves;  // rows per wave
  static_assert(RW % RB == 0, "row batches");
  extern __shared__ float red[];                  // [kLnWaves][2][d]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = d >> 6;
  float pg[NJ], pb[NJ], gg[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    pg[j] = pb[j] = 0.f;
    gg[j] = j < n ? g[lane + 64 * j] : 0.f;
  }
  const int rw0 = blockIdx.x * kLnRowsPerGroup + wave * RW;
  for (int q0 = 0; q0 < RW; q0 += RB) {
    if (rw0 + q0 >= rows) break;  // wave-uniform
    float dv[RB][NJ], xh[RB][NJ], mu[RB], rs[RB];
#pragma unroll
    for (int q = 0; q < RB; ++q) {
      const int r = min(rw0 + q0 + q, rows - 1);  // a short tail repeats the last row
      const int64_t base = (int64_t)r * d + lane;
      mu[q] = mean[r];
      rs[q] = rstd[r];
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        if (j < n) {
          dv[q][j] = (float)dy[base + 64 * j];
          xh[q][j] = (float)xs[base + 64 * j];
        }
    }
#pragma unroll
    for (int q = 0; q < RB; ++q) {
      const int r = rw0 + q0 + q;
      if (r >= rows) break;  // wave-uniform
      const int64_t base = (int64_t)r * d + lane;
      float gy[NJ];
      float s1 = 0.f, s2 = 0.f;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        if (j < n) {
          xh[q][j] = (xh[q][j] - mu[q]) * rs[q];
          gy[j] = dv[q][j] * gg[j];
          s1 += gy[j];
          s2 += gy[j] * xh[q][j];
          pg[j] += dv[q][j] * xh[q][j];
          pb[j] += dv[q][j];
        }
      }
      const float m1 = wave_sum(s1) / (float)d, m2 = wave_sum(s2) / (float)d;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        if (j < n) {
          float o = rs[q] * (gy[j] - m1 - xh[q][j] * m2);
          if (dres) o += (float)dres[base + 64 * j];
          dx[base + 64 * j] = (bf16)o;
        }
      }
    }
  }
#pragma unroll
  for (int j = 0; j < NJ; ++j)
    if (j < n) {
      red[(wave * 2 + 0) * d + lane + 64 * j] = pg[j];
      red[(wave * 2 + 1) * d + lane + 64 * j] = pb[j];
    }
  __syncthreads();
  for (int c = threadIdx.x; c < d; c += blockDim.x) {
    float a = 0.f, bb = 0.f;
    for (int w = 0; w < kLnWaves; ++w) {
      a += red[(w * 2 + 0) * d + c];
      bb += red[(w * 2 + 1) * d + c];
    }
    part[((int64_t)blockIdx.x * 2 + 0) * d + c] = a;
    part[((int64_t)blockIdx.x * 2 + 1) * d + c] = bb;
  }
}

// dg[c] = sum_w part[w][0][c], db[c] = sum_w part[w][1][c] in a fixed
// order: workgroup = 64 columns of one of the two, wave k of 16 sums the
// parts k, k + 16, ... (four accumulators in turn), then the waves add up.
__global__ __launch_bounds__(1024) void ln_param_grad_kernel(const float* __restrict__ part,
                                                             int nparts, int d,
                                                             float* __restrict__ dg,
                                                             float* __restrict__ db) {
  __shared__ float red[16][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c0 = blockIdx.x * 64;  // over the 2 d columns of [dg | db]
  const int which = c0 / d, col = c0 % d + lane;
  const float* src = part + (int64_t)which * d + col;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  int k = 0;
  for (int w = wave; w < nparts; w += 16, ++k) acc[k & 3] += src[(int64_t)w * 2 * d];
  red[wave][lane] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  __syncthreads();
  if (wave == 0) {
    float t = 0.f;
#pragma unroll
    for (int w = 0; w < 16; ++w) t += red[w][lane];
    (which == 0 ? dg : db)[col] = t;
  }
}

// Log-sum-exp of each row of logits from the head product's per-tile
// partials (max, sum of exp(z - max)), one wave per row:
// lse[r] = M + log sum_j s_j exp(m_j - M) with M the largest m_j, and
// row_loss[r] = lse[r] - z[r][target], the target's logit taken again as
// the float32 dot product f[r] . E[target].
__global__ __launch_bounds__(256) void head_lse_kernel(const float* __restrict__ part, int ntile,
                                                       const bf16* __restrict__ f,
                                                       const bf16* __restrict__ E,
                                                       const int32_t* __restrict__ tgt, int rows,
                                                       int d, int V, float* __restrict__ lse,
                                                       float* __restrict__ row_loss) {
  constexpr float kL2e = 1.4426950408889634f;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (r >= rows) return;  // whole waves
  float mx = -INFINITY, sm = 0.f;
  for (int j = lane; j < ntile; j += 64) {
    const float2 q = *reinterpret_cast<const float2*>(part + 2 * ((int64_t)r * ntile + j));
    if (q.x > mx) {
      sm = sm * exp2f((mx - q.x) * kL2e) + q.y;  // exp2f(-inf) = 0 on the first tile
      mx = q.x;
    } else {
      sm += q.y * exp2f((q.x - mx) * kL2e);
    }
  }
  const float M = wave_max(mx);
  const float S = wave_sum(mx == -INFINITY ? 0.f : sm * exp2f((mx - M) * kL2e));
  const float l = M + logf(S);
  const int tk = min(max(tgt[r], 0), V - 1);
  float z = 0.f;
  for (int k = lane; k < d; k += 64)
    z += (float)f[(int64_t)r * d + k] * (float)E[(int64_t)tk * d + k];
  z = wave_sum(z);
  if (lane == 0) {
    lse[r] = l;
    row_loss[r] = l - z;
  }
}

// loss = sum(row_loss) / n, one workgroup, fixed order.
__global__ __launch_bounds__(1024) void loss_sum_kernel(const float* __restrict__ row_loss,
                                                        int n, float* __restrict__ loss) {
  __shared__ float red[16];
  float s = 0.f;
#pragma unroll 4
  for (int i = threadIdx.x; i < n; i += 1024) s += row_loss[i];
  s = wave_sum(s);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = 0.f;
#pragma unroll
    for (int w = 0; w < 16; ++w) t += red[w];
    loss[0] = t / (float)n;
  }
}

// dE[tok[r]] += dx[r] (float32 atomics: rows sharing a token add in any
// order), 8 columns per thread.
__global__ __launch_bounds__(256) void embed_bwd_kernel(const int32_t* __restrict__ tok,
                                                        const bf16* __restrict__ dx,
                                                        float* __restrict__ dE, int rows, int d,
                                                        int V) {
  const int per = d / 8;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)rows * per) return;
  const int r = (int)(i / per), c = (int)(i % per) * 8;
  const int tk = min(max(tok[r], 0), V - 1);
  float v[8];
  ld8(dx + (int64_t)r * d + c, v);
  float* dst = dE + (int64_t)tk * d + c;
#pragma unroll
  for (int k = 0; k < 8; ++k) unsafeAtomicAdd(dst + k, v[k]);
}

// dPe[t] = sum_b dx[b T + t], fixed order.
__global__ __launch_bounds__(256) void pos_bwd_kernel(const bf16* __restrict__ dx,
                                                      float* __restrict__ dPe, int B, int T,
                                                      int d) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)T * d) return;
  float s = 0.f;
  for (int b = 0; b < B; ++b) s += (float)dx[(int64_t)b * T * d + i];
  dPe[i] = s;
}

// AdamW on the flat vectors (decoupled decay, bias-corrected moments) and
// the bf16 working copy of the updated parameters.
__global__ __launch_bounds__(256) void adamw_kernel(float* __restrict__ p,
                                                    const float* __restrict__ g,
                                                    float* __restrict__ m, float* __restrict__ v,
                                                    bf16* __restrict__ pb, int64_t n, float lr,
                                                    float b1, float b2, float eps, float wd,
                                                    float bc1, float bc2) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const float gi = g[i];
    float pi = p[i] * (1.f - lr * wd);
    const float mi = b1 * m[i] + (1.f - b1) * gi;
    const float vi = b2 * v[i] + (1.f - b2) * gi * gi;
    pi -= lr * (mi / bc1) / (sqrtf(vi / bc2) + eps);
    p[i] = pi;
    m[i] = mi;
    v[i] = vi;
    pb[i] = (bf16)pi;
  }
}

__global__ __launch_bounds__(256) void cast_kernel(const float* __restrict__ p,
                                                   bf16* __restrict__ pb, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    pb[i] = (bf16)p[i];
}

unsigned blocks_for(int64_t n, int per_block, int cap) {
  int64_t b = (n + per_block - 1) / per_block;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return (unsigned)b;
}

// ------------------------------------------------------------------ layout

constexpr size_t kAlignB = 256;
size_t upb(size_t x) { return (x + kAlignB - 1) / kAlignB * kAlignB; }

int vocab_padded(int V) { return (V + 127) / 128 * 128; }

// Arrays of the flat parameter vector, in order: E [Vp, d], Pe [T, d]; per
// layer ln1_g, ln1_b [d], Wq, Wk, Wv, Wo, Wm, Wg [d, d], wp [d], ln2_g,
// ln2_b [d], W1 [d, 4d], W2 [4d, d]; lnf_g, lnf_b [d].  Offsets in elements.
constexpr int kLayerArrays = 13;
int model_arrays(const bcmt_model_config& c) { return 2 + kLayerArrays * c.n_layer + 2; }

size_t array_count(const bcmt_model_config& c, int i) {
  const size_t d = c.d;
  if (i == 0) return (size_t)vocab_padded(c.V) * d;
  if (i == 1) return (size_t)c.T * d;
  const int j = i - 2;
  if (j >= kLayerArrays * c.n_layer) return d;  // lnf_g, lnf_b
  switch (j % kLayerArrays) {
    case 2: case 3: case 4: case 5: case 6: case 7: return d * d;
    case 11: return d * 4 * d;
    case 12: return 4 * d * d;
    default: return d;  // LayerNorm gains / biases, wp
  }
}

size_t array_offset(const bcmt_model_config& c, int i) {
  size_t off = 0;
  for (int k = 0; k < i; ++k) off += array_count(c, k);
  return off;
}

struct ModelPlan {
  int BT, d, Vp;
  bcmt_config lc;  // the BCMT layer's config
  size_t layer_saved, layer_ws, wpart_bytes, nparts;
  // offsets into the workspace
  size_t r, a, st1, saved, y, bn, st2, U, A, f, stf, logits, hpart, lse, row_loss;
  size_t dr, dt, df32, dU, dxm, lnpart, wpart, lws, total;

  explicit ModelPlan(const bcmt_model_config& c) {
    BT = c.B * c.T;
    d = c.d;
    Vp = vocab_padded(c.V);
    lc = bcmt_config{c.B, c.T, c.d, c.H, c.L, c.gamma, BCMT_BF16, 0};
    layer_saved = upb(bcmt_saved_bytes(&lc));
    const size_t wf = bcmt_workspace_bytes(&lc, BCMT_PASS_FORWARD);
    const size_t wb = bcmt_workspace_bytes(&lc, BCMT_PASS_BACKWARD);
    layer_ws = upb(wf > wb ? wf : wb);
    nparts = (BT + kLnRowsPerGroup - 1) / kLnRowsPerGroup;
    size_t w = gemm_splitk_partial_bytes(4 * d, d, BT, kWgradMinK);
    const size_t sizes[3] = {gemm_splitk_partial_bytes(d, 4 * d, BT, kWgradMinK),
                             gemm_splitk_partial_bytes(Vp, d, BT, kWgradMinK),
                             gemm_splitk_partial_bytes(BT, d, Vp, kDfMinK)};
    for (size_t x : sizes)
      if (x > w) w = x;
    if (head_partial_bytes(BT, d, Vp) > w) w = head_partial_bytes(BT, d, Vp);
    wpart_bytes = upb(w);
    const size_t act = upb((size_t)BT * d * 2), act4 = upb((size_t)BT * 4 * d * 2);
    const size_t rowf = upb((size_t)BT * 4);
    const int n = c.n_layer;
    size_t off = 0;
    auto take = [&](size_t bytes) {
      const size_t at = off;
      off += upb(bytes);
      return at;
    };
    r = take(act * (2 * n + 1));  // residual stream at every layer boundary
    a = take(act * n);            // LN1 outputs (the layers' inputs)
    st1 = take(rowf * 2 * n);     // LN1 mean, rstd
    saved = take(layer_saved * n);
    y = take(act);                // a layer's output (consumed at once)
    bn = take(act * n);           // LN2 outputs
    st2 = take(rowf * 2 * n);
    U = take(act4 * n);           // MLP pre-activations
    A = take(act4 * n);           // MLP activations
    f = take(act);                // final LayerNorm output
    stf = take(rowf * 2);
    logits = take((size_t)BT * Vp * 2);  // the loss gradient w.r.t. the logits
    hpart = take((size_t)BT * (Vp / 128) * 8);
    lse = take(rowf);
    row_loss = take(rowf);
    dr = take(act);               // gradient of the residual stream
    dt = take(act);
    df32 = take((size_t)BT * d * 4);  // the head's input gradient (float32)
    dU = take(act4);
    dxm = take(act);
    lnpart = take(nparts * 2 * d * 4);
    wpart = take(wpart_bytes);
    lws = take(layer_ws);
    total = off;
  }
};

int check_model(const bcmt_model_config* c) {
  if (!c) return BCMT_ERR_INVALID;
  if (c->V < 2 || c->d < 64 || c->n_layer < 1 || c->B < 1 || c->T < 1 || c->L < 1 || c->H < 1)
    return BCMT_ERR_INVALID;
  if (c->d % 64 != 0 || c->d > 1024 || c->V > 65536) return BCMT_ERR_UNSUPPORTED;
  if ((int64_t)c->B * c->T < 8) return BCMT_ERR_UNSUPPORTED;  // the head product needs 8 rows
  bcmt_config lc{c->B, c->T, c->d, c->H, c->L, c->gamma, BCMT_BF16, 0};
  return bcmt_validate(&lc);
}

bool al16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

}  // namespace
}  // namespace bcmt

using namespace bcmt;

extern "C" {

size_t bcmt_model_param_count(const bcmt_model_config* cfg) {
  if (check_model(cfg) != BCMT_OK) return 0;
  return array_offset(*cfg, model_arrays(*cfg));
}

int bcmt_model_param_array(const bcmt_model_config* cfg, int index, size_t* offset,
                           size_t* count) {
  const int st = check_model(cfg);
  if (st != BCMT_OK) return st;
  if (index < 0 || index >= model_arrays(*cfg) || !offset || !count) return BCMT_ERR_INVALID;
  *offset = array_offset(*cfg, index);
  *count = array_count(*cfg, index);
  return BCMT_OK;
}

size_t bcmt_model_workspace_bytes(const bcmt_model_config* cfg) {
  if (check_model(cfg) != BCMT_OK) return 0;
  return ModelPlan(*cfg).total;
}

int bcmt_model_cast(const bcmt_model_config* cfg, const float* params, void* params_bf16,
                    void* stream) {
  const int st = check_model(cfg);
  if (st != BCMT_OK) return st;
  if (!params || !params_bf16) return BCMT_ERR_INVALID;
  const int64_t n = (int64_t)bcmt_model_param_count(cfg);
  hipLaunchKernelGGL(cast_kernel, dim3(blocks_for(n, 256, 8192)), dim3(256), 0,
                     (hipStream_t)stream, params, (bf16*)params_bf16, n);
  return hipGetLastError() == hipSuccess ? BCMT_OK : BCMT_ERR_HIP;
}

int bcmt_model_train_step(const bcmt_model_config* cfg, const int32_t* tokens,
                          const int32_t* targets, float* params, void* params_bf16,
                          float* grads, float* adam_m, float* adam_v, const bcmt_adamw* opt,
                          float* loss, void* ws, size_t ws_bytes, void* stream,
                          const bcmt_side* side) {
  const int st = check_model(cfg);
  if (st != BCMT_OK) return st;
  if (side && (!side->fork || !side->join)) return BCMT_ERR_INVALID;
  if (!tokens || !targets || !params || !params_bf16 || !grads || !loss || !ws)
    return BCMT_ERR_INVALID;
  if (opt && (!adam_m || !adam_v || opt->step < 1)) return BCMT_ERR_INVALID;
  if (!al16(params) || !al16(params_bf16) || !al16(grads) || !al16(ws) ||
      (opt && (!al16(adam_m) || !al16(adam_v))))
    return BCMT_ERR_INVALID;
  const ModelPlan p(*cfg);
  if (ws_bytes < p.total) return BCMT_ERR_WORKSPACE;
  const bcmt_model_config& c = *cfg;
  hipStream_t s = (hipStream_t)stream;
  char* W = (char*)ws;
  const int BT = p.BT, d = p.d, n = c.n_layer;
  const size_t act = upb((size_t)BT * d * 2), act4 = upb((size_t)BT * 4 * d * 2);
  const size_t rowf = upb((size_t)BT * 4);
  const bf16* PB = (const bf16*)params_bf16;
  auto pw = [&](int i) { return PB + array_offset(c, i); };          // bf16 parameter
  auto pf = [&](int i) { return (const float*)params + array_offset(c, i); };  // float32
  auto gw = [&](int i) { return grads + array_offset(c, i); };        // float32 gradient
  auto lidx = [&](int l, int k) { return 2 + kLayerArrays * l + k; };
  auto R = [&](int k) { return (bf16*)(W + p.r + act * k); };
  auto st1m = [&](int l) { return (float*)(W + p.st1 + rowf * 2 * l); };
  auto st2m = [&](int l) { return (float*)(W + p.st2 + rowf * 2 * l); };
#define CHK(expr)                                        \
  do {                                                   \
    if ((expr) != hipSuccess) return BCMT_ERR_HIP;       \
  } while (0)
#define KCHK()                                           \
  do {                                                   \
    if (hipGetLastError() != hipSuccess) return BCMT_ERR_HIP; \
  } while (0)
  // (The LayerNorm gains and biases are read in float32 from `params`.)
  const unsigned ln_grid = (BT + 3) / 4;
  const unsigned ew_grid = blocks_for((int64_t)BT * (d / 8), 256, 1 << 30);

  // ---- forward
  hipLaunchKernelGGL(embed_fwd_kernel, dim3(ew_grid), dim3(256), 0, s, tokens, pw(0), pw(1), R(0),
                     BT, c.T, d, c.V);
  KCHK();
  for (int l = 0; l < n; ++l) {
    bf16* a = (bf16*)(W + p.a + act * l);
    hipLaunchKernelGGL(add_ln_fwd_kernel, dim3(ln_grid), dim3(256), 0, s, R(2 * l), nullptr,
                       nullptr, pf(lidx(l, 0)), pf(lidx(l, 1)), a, st1m(l), st1m(l) + rowf / 4,
                       BT, d);
    KCHK();
    const bcmt_params lp{pw(lidx(l, 2)), pw(lidx(l, 3)), pw(lidx(l, 4)), pw(lidx(l, 5)),
                         pw(lidx(l, 6)), pw(lidx(l, 7)), pw(lidx(l, 8)), nullptr};
    int e = bcmt_layer_forward(&p.lc, a, &lp, W + p.y, W + p.saved + p.layer_saved * l,
                               W + p.lws, p.layer_ws, s);
    if (e != BCMT_OK) return e;
    bf16* bn = (bf16*)(W + p.bn + act * l);
    hipLaunchKernelGGL(add_ln_fwd_kernel, dim3(ln_grid), dim3(256), 0, s, R(2 * l),
                       (const bf16*)(W + p.y), R(2 * l + 1), pf(lidx(l, 9)), pf(lidx(l, 10)), bn,
                       st2m(l), st2m(l) + rowf / 4, BT, d);
    KCHK();
    bf16* U = (bf16*)(W + p.U + act4 * l);
    bf16* A = (bf16*)(W + p.A + act4 * l);
    {
      GemmDesc g{BT, 4 * d, d, bn, d, false, {pw(lidx(l, 11)), nullptr, nullptr}, 4 * d, true,
                 kSegNone, 0, 1};
      CHK(gemm_gelu(DType::BF16, g, U, A, 4 * d, s));
    }
    {
      GemmDesc g{BT, d, 4 * d, A, 4 * d, false, {pw(lidx(l, 12)), nullptr, nullptr}, d, true,
                 kSegNone, 0, 1};
      CHK(gemm_store(DType::BF16, g, R(2 * l + 2), d, false, R(2 * l + 1), d, s));
    }
  }
  const int lf = 2 + kLayerArrays * n;
  float* stf = (float*)(W + p.stf);
  hipLaunchKernelGGL(add_ln_fwd_kernel, dim3(ln_grid), dim3(256), 0, s, R(2 * n), nullptr, nullptr,
                     pf(lf), pf(lf + 1), (bf16*)(W + p.f), stf, stf + rowf / 4, BT, d);
  KCHK();
  bf16* logits = (bf16*)(W + p.logits);
  float* lse = (float*)(W + p.lse);
  // logits = f E^T: B[k][v] = E[v][k], K-contiguous.  The product is taken
  // twice and never stored: here for each row's log-sum-exp, at the start of
  // the backward for the gradient.
  const GemmDesc head{BT, p.Vp, d, W + p.f, d, false, {pw(0), nullptr, nullptr}, d, false,
                      kSegNone, 0, 1};
  const bool fused_head = head_fused_ok(d, p.Vp);
  int hparts = p.Vp / 128;
  if (fused_head)
    CHK(head_stats(W + p.f, pw(0), BT, d, c.V, p.Vp, (float*)(W + p.hpart), &hparts, s));
  else
    CHK(gemm_head_stats(head, (float*)(W + p.hpart), c.V, s));
  hipLaunchKernelGGL(head_lse_kernel, dim3((BT + 3) / 4), dim3(256), 0, s,
                     (const float*)(W + p.hpart), hparts, (const bf16*)(W + p.f), pw(0),
                     targets, BT, d, c.V, lse, (float*)(W + p.row_loss));
  KCHK();
  hipLaunchKernelGGL(loss_sum_kernel, dim3(1), dim3(1024), 0, s, (const float*)(W + p.row_loss),
                     BT, loss);
  KCHK();

  // ---- backward
  float* wpart = (float*)(W + p.wpart);
  float* lnpart = (float*)(W + p.lnpart);
  bf16* dr = (bf16*)(W + p.dr);
  bf16* dt = (bf16*)(W + p.dt);
  auto ln_bwd = [&](auto dy, const bf16* xs, const float* stats, int gi, const bf16* dres,
                    bf16* dx) -> hipError_t {
    using TY = typename std::remove_cv<typename std::remove_pointer<decltype(dy)>::type>::type;
    const size_t lds = (size_t)kLnWaves * 2 * d * sizeof(float);
    if (d <= 256)
      hipLaunchKernelGGL((ln_bwd_kernel<TY, 4, 4>), dim3((unsigned)p.nparts), dim3(64 * kLnWaves),
                         lds, s, dy, xs, stats, stats + rowf / 4, pf(gi), dres, dx, lnpart, BT, d);
    else
      hipLaunchKernelGGL((ln_bwd_kernel<TY, 16, 1>), dim3((unsigned)p.nparts),
                         dim3(64 * kLnWaves), lds, s, dy, xs, stats, stats + rowf / 4, pf(gi),
                         dres, dx, lnpart, BT, d);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(ln_param_grad_kernel, dim3(2 * d / 64), dim3(1024), 0, s, lnpart,
                       (int)p.nparts, d, gw(gi), gw(gi + 1));
    return hipGetLastError();
  };
  // dlogits = (softmax - onehot) / (B T), over the logits buffer
  // (with the fused head, df = dlogits E comes out of the same pass)
  if (fused_head)
    CHK(head_grad(W + p.f, pw(0), BT, d, c.V, p.Vp, lse, targets, 1.f / (float)BT, logits, p.Vp,
                  wpart, (float*)(W + p.df32), s));
  else
    CHK(gemm_head_grad(head, logits, p.Vp, lse, targets, c.V, 1.f / (float)BT, s));
  {
    // dE = dlogits^T f (the tied head's part; the lookups add below)
    GemmDesc g{p.Vp, d, BT, logits, p.Vp, true, {W + p.f, nullptr, nullptr}, d, true, kSegNone, 0, 1};
    CHK(gemm_splitk(DType::BF16, g, wpart, gw(0), nullptr, nullptr, d, d, false, kWgradMinK, s));
  }
  if (!fused_head) {
    // df = dlogits E: B[v][k] = E[v][k], N-contiguous; K = Vp is long and
    // N = d narrow, so the product is split along K (float32 result)
    GemmDesc g{BT, d, p.Vp, logits, p.Vp, false, {pw(0), nullptr, nullptr}, d, true, kSegNone, 0, 1};
    CHK(gemm_splitk(DType::BF16, g, wpart, (float*)(W + p.df32), nullptr, nullptr, d, d, false,
                    kDfMinK, s));
  }
  CHK(ln_bwd((const float*)(W + p.df32), R(2 * n), stf, lf, nullptr, dr));
  for (int l = n - 1; l >= 0; --l) {
    const bf16* U = (const bf16*)(W + p.U + act4 * l);
    const bf16* A = (const bf16*)(W + p.A + act4 * l);
    const bf16* bn = (const bf16*)(W + p.bn + act * l);
    bf16* dU = (bf16*)(W + p.dU);
    {
      // dU = (dr W2^T) * gelu'(U): B[k][n] = W2[n][k], K-contiguous
      GemmDesc g{BT, 4 * d, d, dr, d, false, {pw(lidx(l, 12)), nullptr, nullptr}, d, false,
                 kSegNone, 0, 1};
      CHK(gemm_gelu_bwd(DType::BF16, g, U, dU, 4 * d, s));
    }
    {
      GemmDesc g{4 * d, d, BT, A, 4 * d, true, {dr, nullptr, nullptr}, d, true, kSegNone, 0, 1};
      CHK(gemm_splitk(DType::BF16, g, wpart, gw(lidx(l, 12)), nullptr, nullptr, d, d, false,
                      kWgradMinK, s));
    }
    {
      GemmDesc g{d, 4 * d, BT, bn, d, true, {dU, nullptr, nullptr}, 4 * d, true, kSegNone, 0, 1};
      CHK(gemm_splitk(DType::BF16, g, wpart, gw(lidx(l, 11)), nullptr, nullptr, 4 * d, 4 * d,
                      false, kWgradMinK, s));
    }
    {
      // d(LN2 out) = dU W1^T: B[k][n] = W1[n][k], K-contiguous
      GemmDesc g{BT, d, 4 * d, dU, 4 * d, false, {pw(lidx(l, 11)), nullptr, nullptr}, 4 * d,
                 false, kSegNone, 0, 1};
      CHK(gemm_store(DType::BF16, g, dt, d, false, nullptr, 0, s));
    }
    CHK(ln_bwd(dt, R(2 * l + 1), st2m(l), lidx(l, 9), dr, dr));
    const bcmt_params lp{pw(lidx(l, 2)), pw(lidx(l, 3)), pw(lidx(l, 4)), pw(lidx(l, 5)),
                         pw(lidx(l, 6)), pw(lidx(l, 7)), pw(lidx(l, 8)), nullptr};
    bcmt_grads lg;
    memset(&lg, 0, sizeof(lg));
    lg.dWq = gw(lidx(l, 2));
    lg.dWk = gw(lidx(l, 3));
    lg.dWv = gw(lidx(l, 4));
    lg.dWo = gw(lidx(l, 5));
    lg.dWm = gw(lidx(l, 6));
    lg.dWg = gw(lidx(l, 7));
    lg.dwp = gw(lidx(l, 8));
    int e = bcmt_layer_backward(&p.lc, W + p.a + act * l, &lp, W + p.saved + p.layer_saved * l,
                                dr, W + p.dxm, &lg, W + p.lws, p.layer_ws, s, side);
    if (e != BCMT_OK) return e;
    CHK(ln_bwd((const bf16*)(W + p.dxm), R(2 * l), st1m(l), lidx(l, 0), dr, dr));
  }
  hipLaunchKernelGGL(embed_bwd_kernel, dim3(ew_grid), dim3(256), 0, s, tokens, dr, gw(0), BT, d,
                     c.V);
  KCHK();
  hipLaunchKernelGGL(pos_bwd_kernel, dim3(blocks_for((int64_t)c.T * d, 256, 1 << 30)), dim3(256),
                     0, s, dr, gw(1), c.B, c.T, d);
  KCHK();

  // ---- optimizer
  if (opt) {
    const int64_t np = (int64_t)bcmt_model_param_count(cfg);
    const float bc1 = 1.f - powf(opt->beta1, (float)opt->step);
    const float bc2 = 1.f - powf(opt->beta2, (float)opt->step);
    hipLaunchKernelGGL(adamw_kernel, dim3(blocks_for(np, 256, 8192)), dim3(256), 0, s, params,
                       grads, adam_m, adam_v, (bf16*)params_bf16, np, opt->lr, opt->beta1,
                       opt->beta2, opt->eps, opt->weight_decay, bc1, bc2);
    KCHK();
  }
#undef CHK
#undef KCHK
  return BCMT_OK;
}

}  // extern "C"
