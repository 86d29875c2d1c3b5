// C ABI of the BCMT layer: argument checks, the buffer plan, and the ordered
// launch sequence of the forward and backward passes.
//
// Forward (Sec. 3.2-3.8 of the paper), all on the caller's stream:
//   1. [Q|K|V] = X [Wq|Wk|Wv]                      matrix cores
//   2. block-local causal attention -> Hcat, lse   matrix cores
//   3. H = Hcat Wo                                 matrix cores
//   4. pooling scores, block softmax -> S          bandwidth
//   5. Q = S Wm (split-K partials)                 matrix cores (N_b rows)
//   6. decayed scans of S and Q -> M, P = M Wm     latency
//   7. U = H Wg; G = sigmoid(U); Y = H + G * P[blk - 1]  (fused epilogue)
// A chunk of a longer sequence (the *_chunk entry points) also takes the
// memory state left by the earlier blocks: before step 5 it is copied into
// `saved` with its memory in the compute type, which is projected by Wm for
// the chunk's first block; the scans start from it and write the state after
// the last block.
// Backward runs the chain rule through the same steps in reverse.  Its
// critical path (gate -> memory -> pooling -> dH -> attention -> dX) stays on
// the caller's stream; the weight-gradient products, which nothing later in
// the pass reads, run on a second stream that the caller may supply: it forks
// from the caller's stream after their inputs exist and joins it before the
// pass ends.  Without one, everything runs on the caller's stream.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <algorithm>
#include <mutex>
#include <vector>

#include "../../include/bcmt.h"
#include "kernels.h"

namespace bcmt {
namespace {

constexpr size_t kAlign = 256;
constexpr int kDh = 64;
constexpr int kMaxD = 2048;

size_t up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Minimum K per split of the D x D weight-gradient products on the side
// stream.  Long inputs (splits of a 512-workgroup plan at least 8192 deep):
// 128, i.e. the plan's two workgroups on every CU.  B = 2, T = 65536,
// D = 1024: 512 instead of 320 workgroups took dW_o and dW_g from 457 to
// 310 us each and the step from 6.49 to 6.23 ms; one workgroup per CU (256)
// took them to 590 us.  Shorter inputs: about 288 workgroups, at least 128
// deep (D = 128: one tile, 128 splits).  At B = 8, T = 1024, D = 768, 468
// workgroups made the products 3.5 us faster but their reductions 1.7 us
// slower and the step 10 us slower (the side stream then crowds out the
// critical path); against 144 workgroups, 288 took the step from 299.3 to
// 298.4-298.9 us.
int dd_min_k(int D, int K) {
  const int64_t tiles = (int64_t)((D + 127) / 128) * ((D + 127) / 128);
  if ((int64_t)K * tiles / 512 >= 8192) return 128;
  const int mk = (int)((K * tiles / 288 + 63) / 64 * 64);
  return mk < 128 ? 128 : mk;
}
// The same for dW_{q,k,v}: splits at least 128 deep (4 at D = 768, where
// 2 were slower; up to 128 at small D).
constexpr int kQkvMinK = 128;

struct Plan {
  int B, T, D, H, L, nb;
  size_t es;
  DType dt;
  // saved (forward -> backward)
  size_t qkv, o, lse, h, g, s, stats, S, M, Mt, P;
  size_t cN, cZ, cMt, cP;  // incoming chunk state: N, Z, N / Z (compute type), (N / Z) Wm
  size_t saved_bytes;
  // forward scratch
  size_t sp, St, mpart, cpart, fwd_bytes;
  // backward scratch
  size_t du, pbar, pbar_lo, dS, dM, mpart_b, a, ds, dwpp, dh, dout, delta, dqkv, wpart;
  size_t cpbar, cpbar_lo, cdm, ce0, cpart_b;  // chunk state gradients
  size_t dgp;  // decay-gradient partials (dgp_rows + B rows)
  int dgp_rows;
  size_t bwd_bytes;

  explicit Plan(const bcmt_config& c) {
    B = c.B;
    T = c.T;
    D = c.D;
    H = c.H;
    L = c.L;
    nb = (T + L - 1) / L;
    dt = c.dtype == BCMT_BF16 ? DType::BF16 : DType::F32;
    es = dt == DType::BF16 ? 2 : 4;
    const size_t BT = (size_t)B * T, BTD = BT * D, BND = (size_t)B * nb * D;
    size_t off = 0;
    auto take = [&](size_t bytes) {
      size_t at = off;
      off += up(bytes);
      return at;
    };
    qkv = take(3 * BTD * es);
    o = take(BTD * es);
    lse = take((size_t)B * H * T * 4);
    h = take(BTD * es);
    g = take(BTD * es);
    s = take(BT * 4);
    stats = take((size_t)B * nb * 2 * 4);
    S = take(BND * 4);
    M = take(BND * 4);
    Mt = take(BND * es);
    P = take(BND * 4);
    const size_t BD = (size_t)B * D;
    cN = take(BD * 4);
    cZ = take(BD * 4);  // one normaliser per sequence, or per channel
    cMt = take(BD * es);
    cP = take(BD * 4);
    saved_bytes = off;

    off = 0;
    sp = take(BT * (D / kDh) * 4);  // partial pooling scores, D / 64 per token
    St = take(BND * es);
    const bool pc = c.flags & BCMT_FLAG_CHANNEL_DECAY;
    mpart = take(mem_part_bytes(B, nb, D, pc));  // W_m product partials (scan + product path)
    cpart = take(carry_part_bytes(B, D));
    fwd_bytes = off;

    off = 0;
    du = take(BTD * es);
    // the shifted context gradient; bf16 keeps each value as hi + lo, a row
    // [hi (D) | lo (D)] (so that one product over 2D takes both)
    pbar = take(BND * es * (dt == DType::BF16 ? 2 : 1));
    pbar_lo = pbar + (dt == DType::BF16 ? (size_t)D * es : 0);
    dS = take(BND * 4);
    dM = take(0);  // (the long path's dM stays in split-K partials)
    mpart_b = take(mem_part_bytes(B, nb, D, pc));
    a = take(BT * 4);
    ds = take(BT * 4);
    dwpp = take((size_t)pool_bwd_partial_rows(dt, B, T, D, L) * D * 4);
    dh = take(BTD * es);
    dout = take(BTD * es);
    delta = take((size_t)B * H * T * 4);
    dqkv = take(3 * BTD * es);
    {
      const int BTi = B * T, BNi = B * nb;
      size_t w = gemm_splitk_partial_bytes(D, 3 * D, BTi, kQkvMinK);
      w = std::max(w, gemm_splitk_partial_bytes(D, D, BTi, dd_min_k(D, BTi)));
      w = std::max(w, gemm_wgrad_partial_bytes(D, D, BNi));
      wpart = take(w);  // weight gradients (side stream, one after another)
    }
    cpbar = take(BD * es);
    cpbar_lo = take(dt == DType::BF16 ? BD * es : 0);
    cdm = take(BD * 4);
    ce0 = take(BD * 4);
    cpart_b = take(carry_part_bytes(B, D));
    // decay-gradient partials: the memory backward's rows, then B rows of
    // the chunked path's first-block terms
    dgp_rows = dg_part_rows(B, nb, D, pc);
    dgp = take((size_t)(dgp_rows + B) * (pc ? D : 1) * 4);
    bwd_bytes = off;
  }
};

// Decode state (the current block's caches and the memory state) and the
// scratch of one decode step.
struct DecPlan {
  int B, D, H, L;
  DType dt;
  size_t es;
  size_t Kc, Vc, Hc, spc, N, Z, C, state_bytes;
  size_t o, Mt, part, cpart, ws_bytes;

  explicit DecPlan(const bcmt_config& c) {
    B = c.B;
    D = c.D;
    H = c.H;
    L = c.L;
    dt = c.dtype == BCMT_BF16 ? DType::BF16 : DType::F32;
    es = dt == DType::BF16 ? 2 : 4;
    const size_t BLD = (size_t)B * L * D, BD = (size_t)B * D;
    size_t off = 0;
    auto take = [&](size_t bytes) {
      size_t at = off;
      off += up(bytes);
      return at;
    };
    Kc = take(BLD * es);
    Vc = take(BLD * es);
    Hc = take(BLD * es);
    spc = take((size_t)B * L * dec_score_parts(D) * 4);
    N = take(BD * 4);
    Z = take(BD * 4);  // one normaliser per sequence, or per channel
    C = take(BD * 4);
    state_bytes = off;
    off = 0;
    o = take(BD * es);
    Mt = take(BD * es);
    part = take(dec_part_bytes(dt, B, D));
    cpart = take(carry_part_bytes(B, D));
    ws_bytes = off;
  }
};

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int check_config(const bcmt_config* c) {
  if (!c) return BCMT_ERR_INVALID;
  if (c->B < 1 || c->T < 1 || c->D < 1 || c->H < 1 || c->L < 1) return BCMT_ERR_INVALID;
  if (c->D % c->H != 0) return BCMT_ERR_INVALID;
  if (!(c->gamma >= 0.0f && c->gamma < 1.0f)) return BCMT_ERR_INVALID;
  if (c->dtype != BCMT_F32 && c->dtype != BCMT_BF16) return BCMT_ERR_INVALID;
  if (c->flags & ~(BCMT_FLAG_RESIDUAL | BCMT_FLAG_ACCUM_WGRAD | BCMT_FLAG_CHANNEL_DECAY))
    return BCMT_ERR_INVALID;
  // Heads of 64 dimensions (matrix-core attention) or of 16 / 32 (the
  // paper's model width); D a multiple of 64 for the 64-column score parts.
  const int dh = c->D / c->H;
  if ((dh != kDh && dh != 16 && dh != 32) || c->D % 64 != 0 || c->D > kMaxD)
    return BCMT_ERR_UNSUPPORTED;
  // Grid limits: rows of the projections, blocks, batch * heads.
  const int64_t BT = (int64_t)c->B * c->T;
  const int64_t nb = ((int64_t)c->T + c->L - 1) / c->L;
  if (BT > 65535LL * 128 || nb > 65535 || (int64_t)c->B * c->H > 65535 || c->B > 65535)
    return BCMT_ERR_UNSUPPORTED;
  return BCMT_OK;
}

bool overlaps(const void* a, const void* b, size_t n) {
  const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + n && y < x + n;
}

int check_decode(const bcmt_config* c) {
  const int st = check_config(c);
  if (st != BCMT_OK) return st;
  if (c->L > dec_max_blocklen() || c->B > dec_max_batch() || c->D / c->H != kDh)
    return BCMT_ERR_UNSUPPORTED;
  return BCMT_OK;
}

// The per-channel decay of a config with BCMT_FLAG_CHANNEL_DECAY (null
// otherwise); such a config needs it, 4-byte aligned.
const float* channel_decay(const bcmt_config* c, const bcmt_params* prm) {
  return (c->flags & BCMT_FLAG_CHANNEL_DECAY) ? prm->gamma_ch : nullptr;
}
bool decay_ok(const bcmt_config* c, const bcmt_params* prm) {
  if (!(c->flags & BCMT_FLAG_CHANNEL_DECAY)) return true;
  return prm->gamma_ch && ((uintptr_t)prm->gamma_ch & 3u) == 0;
}

// A chunk state, when given, needs both members: N 16-byte and Z 4-byte aligned.
bool carry_ok(const bcmt_carry* c) {
  if (!c) return true;
  return c->N && c->Z && aligned16(c->N) && ((uintptr_t)c->Z & 3u) == 0;
}


// ------------------------------------------------------------------ tracing
// Named stages of the two passes; each is one kernel launch.
enum Stage {
  ST_QKV, ST_ATTN_FWD, ST_WO, ST_POOL_FWD, ST_CARRY_IN, ST_CARRY_PROJ, ST_WM_FWD, ST_SCAN_FWD,
  ST_GATE,
  ST_GATE_BWD, ST_WG_WGRAD, ST_WG_WGRAD_RED, ST_WM_WGRAD,
  ST_WM_WGRAD_RED, ST_CARRY_WGRAD, ST_CARRY_DGRAD, ST_WM_BWD, ST_MEM_BWD, ST_CARRY_BWD,
  ST_POOL_BWD, ST_DWP,
  ST_DGAMMA,
  ST_HBAR, ST_WO_DGRAD, ST_WO_WGRAD, ST_WO_WGRAD_RED,
  ST_ATTN_BWD_BLOCK, ST_ATTN_BWD_DQ, ST_ATTN_BWD_DKDV, ST_DX, ST_QKV_WGRAD, ST_QKV_WGRAD_RED,
  ST_DEC_RESET, ST_DEC_QKV, ST_DEC_ATTN, ST_DEC_WO, ST_DEC_WO_FIN, ST_DEC_GATE, ST_DEC_GATE_FIN,
  ST_DEC_POOL, ST_DEC_MEM, ST_DEC_MEM_FIN,
  ST_COUNT
};
const char* const kStageNames[ST_COUNT] = {
    "fwd.qkv_gemm", "fwd.attention", "fwd.wo_gemm", "fwd.pool", "fwd.carry_in",
    "fwd.carry_proj_gemm", "fwd.wm_gemm", "fwd.memory_scan",
    "fwd.gate_gemm", "bwd.gate", "bwd.wg_wgrad_gemm", "bwd.wg_wgrad_reduce",
    "bwd.wm_wgrad_gemm", "bwd.wm_wgrad_reduce", "bwd.carry_wm_wgrad_gemm",
    "bwd.carry_dgrad_gemm", "bwd.wm_dgrad_gemm", "bwd.memory_scan", "bwd.carry_in", "bwd.pool", "bwd.pool_dwp",
    "bwd.decay_grad",
    "bwd.wg_dgrad_gemm",
    "bwd.wo_dgrad_gemm", "bwd.wo_wgrad_gemm", "bwd.wo_wgrad_reduce", "bwd.attention_block", "bwd.attention_dq",
    "bwd.attention_dkdv", "bwd.qkv_dgrad_gemm", "bwd.qkv_wgrad_gemm", "bwd.qkv_wgrad_reduce",
    "dec.reset", "dec.qkv_gemv", "dec.attention", "dec.wo_gemv", "dec.wo_finish",
    "dec.gate_gemv", "dec.gate_finish", "dec.pool", "dec.wm_gemv", "dec.wm_finish"};

struct Tracer {
  std::atomic<bool> on{false};
  std::mutex mu;
  struct Rec {
    int stage;
    hipEvent_t a, b;
  };
  std::vector<Rec> pending;
  // Events are created by bcmt_trace_enable only, never by a layer call; a
  // launch that finds the pool empty is not timed (and counted as dropped).
  std::vector<hipEvent_t> pool;
  int created = 0;
  int64_t dropped = 0;
  double total[ST_COUNT] = {};
  int calls[ST_COUNT] = {};

  hipEvent_t take() {
    if (pool.empty()) {
      ++dropped;
      return nullptr;
    }
    hipEvent_t e = pool.back();
    pool.pop_back();
    return e;
  }
};
Tracer g_trace;
// Events the tracer holds: two per traced launch, enough for a few hundred
// passes between two reads.
constexpr int kTraceEvents = 16384;

// Brackets one launch with two events on the launch stream when tracing is on.
struct TraceScope {
  int stage;
  hipStream_t s;
  hipEvent_t a = nullptr;
  TraceScope(int st, hipStream_t str) : stage(st), s(str) {
    if (!g_trace.on.load(std::memory_order_relaxed)) return;
    std::lock_guard<std::mutex> lk(g_trace.mu);
    if (g_trace.pool.size() < 2) {
      ++g_trace.dropped;
      return;
    }
    a = g_trace.take();
    if (a && hipEventRecord(a, s) != hipSuccess) {
      g_trace.pool.push_back(a);
      a = nullptr;
    }
  }
  void done() {
    if (!a) return;
    std::lock_guard<std::mutex> lk(g_trace.mu);
    hipEvent_t b = g_trace.take();
    if (b && hipEventRecord(b, s) == hipSuccess) {
      g_trace.pending.push_back({stage, a, b});
    } else {
      g_trace.pool.push_back(a);
      if (b) g_trace.pool.push_back(b);
    }
    a = nullptr;
  }
};

// Makes `to` wait for everything enqueued so far on `from`.
hipError_t order_after(hipStream_t to, hipStream_t from, hipEvent_t e) {
  hipError_t r = hipEventRecord(e, from);
  if (r != hipSuccess) return r;
  return hipStreamWaitEvent(to, e, 0);
}

// A split-K product and its reduction as two traced stages.
#define LAUNCH_SPLITK(stage, stage_red, dt, g, part, C0, C1, C2, ldc, seg, acc, min_k)           \
  do {                                                                                        \
    int sp_ = 0;                                                                              \
    LAUNCH(stage, gemm_splitk_product(dt, g, part, C0, C1, C2, ldc, seg, acc, min_k, &sp_, s)); \
    if (sp_ > 1)                                                                              \
      LAUNCH(stage_red, gemm_splitk_reduce(part, sp_, (g).M, (g).N, C0, C1, C2, ldc, seg, acc, s)); \
  } while (0)


#define LAUNCH(stage, expr)                            \
  do {                                                 \
    TraceScope ts_(stage, s);                          \
    if ((expr) != hipSuccess) return BCMT_ERR_HIP;     \
    ts_.done();                                        \
  } while (0)

}  // namespace
}  // namespace bcmt

using namespace bcmt;

extern "C" {

int bcmt_validate(const bcmt_config* cfg) { return check_config(cfg); }

size_t bcmt_saved_bytes(const bcmt_config* cfg) {
  if (check_config(cfg) != BCMT_OK) return 0;
  return Plan(*cfg).saved_bytes;
}

size_t bcmt_workspace_bytes(const bcmt_config* cfg, int pass) {
  if (check_config(cfg) != BCMT_OK) return 0;
  Plan p(*cfg);
  switch (pass) {
    case BCMT_PASS_FORWARD: return p.fwd_bytes;
    case BCMT_PASS_INFERENCE: return p.fwd_bytes + p.saved_bytes;
    case BCMT_PASS_BACKWARD: return p.bwd_bytes;
    default: return 0;
  }
}

const char* bcmt_strerror(int status) {
  switch (status) {
    case BCMT_OK: return "ok";
    case BCMT_ERR_INVALID: return "invalid argument";
    case BCMT_ERR_UNSUPPORTED: return "configuration not supported by the GPU path";
    case BCMT_ERR_WORKSPACE: return "workspace too small";
    case BCMT_ERR_HIP: return "HIP launch failed";
    default: return "unknown status";
  }
}

int bcmt_version(void) { return 20100; }

int bcmt_side_events_create(bcmt_side* side) {
  if (!side) return BCMT_ERR_INVALID;
  side->fork = side->join = nullptr;
  const unsigned flags = hipEventDisableTiming | hipEventDisableSystemFence;
  hipEvent_t f = nullptr, j = nullptr;
  if (hipEventCreateWithFlags(&f, flags) != hipSuccess) return BCMT_ERR_HIP;
  if (hipEventCreateWithFlags(&j, flags) != hipSuccess) {
    (void)hipEventDestroy(f);
    return BCMT_ERR_HIP;
  }
  side->fork = f;
  side->join = j;
  return BCMT_OK;
}

int bcmt_side_events_destroy(bcmt_side* side) {
  if (!side) return BCMT_ERR_INVALID;
  int st = BCMT_OK;
  for (void** e : {&side->fork, &side->join}) {
    if (*e && hipEventDestroy((hipEvent_t)*e) != hipSuccess) st = BCMT_ERR_HIP;
    *e = nullptr;
  }
  return st;
}

int bcmt_trace_enable(int on) {
  if (on) {
    // The timing events are created here, on the current device, once.
    std::lock_guard<std::mutex> lk(g_trace.mu);
    while (g_trace.created < kTraceEvents) {
      hipEvent_t e = nullptr;
      if (hipEventCreate(&e) != hipSuccess) break;
      g_trace.pool.push_back(e);
      ++g_trace.created;
    }
  }
  return g_trace.on.exchange(on != 0) ? 1 : 0;
}

int bcmt_trace_read(bcmt_trace_entry* out, int max_entries) {
  if (max_entries < 0 || (max_entries > 0 && !out)) return BCMT_ERR_INVALID;
  std::lock_guard<std::mutex> lk(g_trace.mu);
  int st = BCMT_OK;
  for (auto& r : g_trace.pending) {
    float ms = 0.f;
    if (hipEventSynchronize(r.b) != hipSuccess || hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) {
      st = BCMT_ERR_HIP;
    } else {
      g_trace.total[r.stage] += ms;
      g_trace.calls[r.stage] += 1;
    }
    g_trace.pool.push_back(r.a);
    g_trace.pool.push_back(r.b);
  }
  g_trace.pending.clear();
  if (st != BCMT_OK) return st;
  int n = 0;
  for (int k = 0; k < ST_COUNT; ++k) {
    if (g_trace.calls[k] == 0) continue;
    if (n < max_entries) {
      out[n].name = kStageNames[k];
      out[n].calls = g_trace.calls[k];
      out[n].total_ms = g_trace.total[k];
    }
    ++n;
    g_trace.calls[k] = 0;
    g_trace.total[k] = 0.0;
  }
  return n;
}

}  // extern "C"

// The forward and backward passes; `chunk` selects the chunked form, with an
// incoming and an outgoing memory state.
static int layer_forward(const bcmt_config* cfg, const void* X, const bcmt_params* prm, void* Y,
                         void* saved, void* ws, size_t ws_bytes, void* stream, bool chunk,
                         const bcmt_carry* cin, const bcmt_carry* cout) {
  int st = check_config(cfg);
  if (st != BCMT_OK) return st;
  if (!X || !prm || !Y) return BCMT_ERR_INVALID;
  if (!carry_ok(cin) || !carry_ok(cout) || !decay_ok(cfg, prm)) return BCMT_ERR_INVALID;
  const void* w[7] = {prm->Wq, prm->Wk, prm->Wv, prm->Wo, prm->Wm, prm->Wg, prm->wp};
  for (const void* p : w)
    if (!p || !aligned16(p)) return BCMT_ERR_INVALID;
  if (!aligned16(X) || !aligned16(Y) || (saved && !aligned16(saved)) || (ws && !aligned16(ws)))
    return BCMT_ERR_INVALID;
  Plan p(*cfg);
  const size_t act = (size_t)p.B * p.T * p.D * p.es;
  if (overlaps(X, Y, act)) return BCMT_ERR_INVALID;
  const size_t need = saved ? p.fwd_bytes : p.fwd_bytes + p.saved_bytes;
  if (!ws) return BCMT_ERR_INVALID;
  if (ws_bytes < need) return BCMT_ERR_WORKSPACE;

  hipStream_t s = (hipStream_t)stream;
  char* W = (char*)ws;
  char* SV = saved ? (char*)saved : W + p.fwd_bytes;
  const int BT = p.B * p.T, D = p.D;
  const DType dt = p.dt;

  // 1. Q | K | V projections (Sec. 3.3).
  {
    GemmDesc g{BT, 3 * D, D, X, D, false, {prm->Wq, prm->Wk, prm->Wv}, D, true, kSegN, D, 1};
    LAUNCH(ST_QKV, gemm_store(dt, g, SV + p.qkv, 3 * D, false, nullptr, 0, s));
  }
  // 2. Block-local causal attention (Sec. 3.3, 3.6).
  LAUNCH(ST_ATTN_FWD, attn_fwd(dt, SV + p.qkv, SV + p.o, (float*)(SV + p.lse), p.B, p.T, D, p.H, p.L, s));
  // One block and no earlier state: the memory is empty, so C = 0 and
  // Y = H (+X) exactly (Sec. 3.5, 3.8); the pooling, the scan and the gate
  // product would only compute terms that vanish.
  if (p.nb == 1 && !chunk) {
    GemmDesc g{BT, D, D, SV + p.o, D, false, {prm->Wo, nullptr, nullptr}, D, true, kSegNone, 0, 1};
    LAUNCH(ST_WO, gemm_store(dt, g, Y, D, false, (cfg->flags & BCMT_FLAG_RESIDUAL) ? X : nullptr,
                             D, s));
    return BCMT_OK;
  }
  // 3. Output projection (Sec. 3.3), also writing partial pooling scores.
  {
    GemmDesc g{BT, D, D, SV + p.o, D, false, {prm->Wo, nullptr, nullptr}, D, true, kSegNone, 0, 1};
    LAUNCH(ST_WO, gemm_score(dt, g, SV + p.h, prm->wp, (float*)(W + p.sp), s));
  }
  // 4. Adaptive summaries (Sec. 3.4); the launch also clears the records of
  // the look-back scan that follows (long sequences, few of them).
  int64_t nflag = 0;
  float* flags = mem_lb_flags((float*)(W + p.mpart), p.B, p.nb, D,
                              channel_decay(cfg, prm) != nullptr, chunk, &nflag);
  LAUNCH(ST_POOL_FWD, pool_fwd(dt, SV + p.h, (const float*)(W + p.sp), D / kDh,
                               (float*)(SV + p.s), (float*)(SV + p.S), W + p.St,
                               (float*)(SV + p.stats), p.B, p.T, D, p.L, flags, nflag, s));
  // 5-6. Exponential memory and its projection (Sec. 3.5): one kernel
  // projects the summaries (Q = S Wm, over only B * N_b rows) and scans S
  // and Q, which yields M and P = M Wm (the decayed sum is linear); the
  // shift is applied where P is read.  A chunk first takes the state of the
  // earlier blocks (a copy, so that carry_out may overwrite carry_in) and
  // projects its memory for the first block.
  Carry cr;
  cr.gvec = channel_decay(cfg, prm);
  cr.zcol = cr.gvec != nullptr;
  if (chunk) {
    LAUNCH(ST_CARRY_IN, carry_prep(dt, cin ? cin->N : nullptr, cin ? cin->Z : nullptr,
                                   (float*)(SV + p.cN), (float*)(SV + p.cZ), SV + p.cMt,
                                   cin ? nullptr : (float*)(SV + p.cP), p.B, D, cr.zcol, s));
    if (cin)
      LAUNCH(ST_CARRY_PROJ, carry_proj(dt, SV + p.cMt, prm->Wm, (float*)(SV + p.cP),
                                       (float*)(W + p.cpart), false, false, p.B, D, s));
    cr.Nin = (const float*)(SV + p.cN);
    cr.Zin = (const float*)(SV + p.cZ);
    cr.Pc = (const float*)(SV + p.cP);
    cr.Nout = cout ? cout->N : nullptr;
    cr.Zout = cout ? cout->Z : nullptr;
  }
  if (mem_fused(p.nb, cr.gvec != nullptr)) {
    LAUNCH(ST_SCAN_FWD, mem_fwd(dt, W + p.St, prm->Wm, (const float*)(SV + p.S),
                                (float*)(SV + p.M), SV + p.Mt, (float*)(SV + p.P),
                                (float*)(W + p.mpart), p.B, p.nb, D, cfg->gamma, cr, s));
  } else {
    // the W_m product and the scans timed apart
    const bool pc = cr.gvec != nullptr;
    int nq = 0;
    if (!pc)
      LAUNCH(ST_WM_FWD, mem_fwd_proj(dt, W + p.St, prm->Wm, SV + p.Mt, (float*)(SV + p.P),
                                     (float*)(W + p.mpart), p.B, p.nb, D, false, &nq, s));
    LAUNCH(ST_SCAN_FWD, mem_fwd_scan(dt, (const float*)(SV + p.S), (float*)(SV + p.M), SV + p.Mt,
                                     (float*)(SV + p.P), (float*)(W + p.mpart), nq, p.B, p.nb, D,
                                     cfg->gamma, cr, s));
    if (pc)
      LAUNCH(ST_WM_FWD, mem_fwd_proj(dt, W + p.St, prm->Wm, SV + p.Mt, (float*)(SV + p.P),
                                     (float*)(W + p.mpart), p.B, p.nb, D, true, &nq, s));
  }
  // 7. Gate and injection (Sec. 3.7, 3.8).
  {
    GemmDesc g{BT, D, D, SV + p.h, D, false, {prm->Wg, nullptr, nullptr}, D, true, kSegNone, 0, 1};
    GateEpi e{Y, SV + p.g, SV + p.h, (cfg->flags & BCMT_FLAG_RESIDUAL) ? X : nullptr,
              (const float*)(SV + p.P), p.T, p.L, p.nb, D,
              chunk ? (const float*)(SV + p.cP) : nullptr};
    LAUNCH(ST_GATE, gemm_gate(dt, g, e, s));
  }
  return BCMT_OK;
}

static int layer_backward(const bcmt_config* cfg, const void* X, const bcmt_params* prm,
                          const void* saved, const void* dY, void* dX, const bcmt_grads* grads,
                          void* ws, size_t ws_bytes, void* stream, const bcmt_side* side,
                          bool chunk, const bcmt_carry* dcout, const bcmt_carry* dcin) {
  int st = check_config(cfg);
  if (st != BCMT_OK) return st;
  if (!X || !prm || !saved || !dY) return BCMT_ERR_INVALID;
  if (side && (!side->fork || !side->join)) return BCMT_ERR_INVALID;
  if (!carry_ok(dcout) || !carry_ok(dcin) || !decay_ok(cfg, prm)) return BCMT_ERR_INVALID;
  const void* w[7] = {prm->Wq, prm->Wk, prm->Wv, prm->Wo, prm->Wm, prm->Wg, prm->wp};
  for (const void* p : w)
    if (!p || !aligned16(p)) return BCMT_ERR_INVALID;
  if (!aligned16(X) || !aligned16(saved) || !aligned16(dY) || (dX && !aligned16(dX)) ||
      (ws && !aligned16(ws)))
    return BCMT_ERR_INVALID;
  bcmt_grads none;
  memset(&none, 0, sizeof(none));
  const bcmt_grads& gr = grads ? *grads : none;
  const float* gp[7] = {gr.dWq, gr.dWk, gr.dWv, gr.dWo, gr.dWm, gr.dWg, gr.dwp};
  for (const float* q : gp)
    if (q && !aligned16(q)) return BCMT_ERR_INVALID;
  if (gr.dgamma && ((uintptr_t)gr.dgamma & 3u)) return BCMT_ERR_INVALID;
  const float* gvec = channel_decay(cfg, prm);
  if (gvec && gr.dgamma_ch && ((uintptr_t)gr.dgamma_ch & 3u)) return BCMT_ERR_INVALID;
  // the decay gradient: one scalar, or one value per channel
  float* dgam = gvec ? gr.dgamma_ch : gr.dgamma;
  Plan p(*cfg);
  const int dgr = dg_part_rows_used(p.B, p.nb, p.D, gvec != nullptr, chunk);  // rows this call writes
  const size_t act = (size_t)p.B * p.T * p.D * p.es;
  if (dX && (overlaps(dX, dY, act) || overlaps(dX, X, act))) return BCMT_ERR_INVALID;
  if (!ws) return BCMT_ERR_INVALID;
  if (ws_bytes < p.bwd_bytes) return BCMT_ERR_WORKSPACE;

  // The weight-gradient products go to the caller's second stream when one
  // is given.  With per-stage tracing on, everything runs on the caller's
  // stream so that each stage is timed alone.
  const bool fork = side && !g_trace.on.load(std::memory_order_relaxed);
  const hipStream_t main_s = (hipStream_t)stream;
  const hipStream_t side_s = fork ? (hipStream_t)side->stream : main_s;
  const hipEvent_t ev_fork = fork ? (hipEvent_t)side->fork : nullptr;
  const hipEvent_t ev_join = fork ? (hipEvent_t)side->join : nullptr;
  hipStream_t s = main_s;  // the stream LAUNCH enqueues on
  const char* SV = (const char*)saved;
  char* W = (char*)ws;
  const int BT = p.B * p.T, D = p.D, BN = p.B * p.nb;
  const DType dt = p.dt;
  const bool residual = cfg->flags & BCMT_FLAG_RESIDUAL;

  const bool accum = cfg->flags & BCMT_FLAG_ACCUM_WGRAD;
  float* wpart = (float*)(W + p.wpart);
  int nfork = 0;
  // Work between SIDE_BEGIN and SIDE_END runs on the second stream, after
  // everything enqueued so far on the caller's stream.  One fork event serves
  // every fork: each wait takes the record made just before it.
#define SIDE_BEGIN()                                                                   \
  do {                                                                                 \
    if (fork && order_after(side_s, main_s, ev_fork) != hipSuccess) return BCMT_ERR_HIP; \
    nfork += fork;                                                                     \
    s = side_s;                                                                        \
  } while (0)
#define SIDE_END() (s = main_s)
  const bool single = p.nb == 1 && !chunk;
  if (single) {
    // One block, no earlier state: Y = H (+X), so dH = dY, and dW_g, dW_m,
    // dw_p and the decay gradient are zero (written unless accumulating).
    if (!accum && (gr.dWg || gr.dWm || gr.dwp || dgam)) {
      SIDE_BEGIN();
      LAUNCH(ST_GATE_BWD, fill_f32(gr.dWg, gr.dWg ? (int64_t)D * D : 0, 0.f, s));
      LAUNCH(ST_GATE_BWD, fill_f32(gr.dWm, gr.dWm ? (int64_t)D * D : 0, 0.f, s));
      LAUNCH(ST_GATE_BWD, fill_f32(gr.dwp, gr.dwp ? D : 0, 0.f, s));
      LAUNCH(ST_GATE_BWD, fill_f32(dgam, dgam ? (gvec ? D : 1) : 0, 0.f, s));
      SIDE_END();
    }
  }
  const void* dH = single ? dY : (const void*)(W + p.dh);
  if (!single) {
    // Gate and injection: dU, and the block sums of dY * G shifted back by one.
    // The weight matrices, dwp and the decay gradient are written (or
    // accumulated) by fixed-order reductions.
    const bool lo = dt == DType::BF16;  // context gradients kept as hi + lo
    // (also clearing the records of the look-back scan of the memory
    // backward: fewer than 128 sequence x column slices, at most 64 segments
    // of 128 words each, so the count fits an int)
    int64_t nflag = 0;
    float* flags = mem_lb_flags((float*)(W + p.mpart_b), p.B, p.nb, D, gvec != nullptr, chunk,
                                &nflag);
    LAUNCH(ST_GATE_BWD, gate_bwd(dt, dY, SV + p.g, (const float*)(SV + p.P), W + p.du, W + p.pbar,
                                 lo ? W + p.pbar_lo : nullptr, flags, (int)nflag, nullptr, p.B,
                                 p.T, D, p.L,
                                 chunk ? (const float*)(SV + p.cP) : nullptr,
                                 chunk ? W + p.cpbar : nullptr,
                                 (chunk && lo) ? W + p.cpbar_lo : nullptr, s));
    // dWg = H^T dU and dWm = M^T dP on the side stream.
    if (gr.dWg || gr.dWm) {
      SIDE_BEGIN();
      {
        if (gr.dWg) {
          GemmDesc g{D, D, BT, SV + p.h, D, true, {W + p.du, nullptr, nullptr}, D, true, kSegNone, 0, 1};
          LAUNCH_SPLITK(ST_WG_WGRAD, ST_WG_WGRAD_RED, dt, g, wpart, gr.dWg, nullptr, nullptr, D, D,
                        accum, dd_min_k(D, BT));
        }
        if (gr.dWm) {
          GemmDesc g{D, D, BN, SV + p.Mt, D, true, {W + p.pbar, nullptr, nullptr},
                     lo ? 2 * D : D, true, kSegNone, 0, 1};
          LAUNCH_SPLITK(ST_WM_WGRAD, ST_WM_WGRAD_RED, dt, g, wpart, gr.dWm, nullptr, nullptr, D, D,
                        accum, 512);
          if (chunk) {
            // The earlier blocks' memory fed the first block: dWm += Mc^T dPc.
            GemmDesc gc{D, D, p.B, SV + p.cMt, D, true, {W + p.cpbar, nullptr, nullptr}, D, true,
                        kSegNone, 0, 1};
            LAUNCH_SPLITK(ST_CARRY_WGRAD, ST_CARRY_WGRAD, dt, gc, wpart, gr.dWm, nullptr, nullptr,
                          D, D, true, 512);
          }
        }
      }
      SIDE_END();
    }
    // Memory projection and decayed reverse scan: dM = dP Wm^T, dS and the
    // decay gradient, in one kernel.  A chunk also feeds in the gradient of
    // the state it passed on and forms the gradient of the state it took.
    Carry cr;
    cr.gvec = gvec;
    cr.zcol = gvec != nullptr;
    if (chunk) {
      LAUNCH(ST_CARRY_DGRAD, carry_proj(dt, W + p.cpbar, prm->Wm, (float*)(W + p.cdm),
                                        (float*)(W + p.cpart_b), true, false, p.B, D, s));
      if (lo)
        LAUNCH(ST_CARRY_DGRAD, carry_proj(dt, W + p.cpbar_lo, prm->Wm, (float*)(W + p.cdm),
                                          (float*)(W + p.cpart_b), true, true, p.B, D, s));
      cr.Zin = (const float*)(SV + p.cZ);
      cr.dNout = dcout ? dcout->N : nullptr;
      cr.dZout = dcout ? dcout->Z : nullptr;
      cr.e0 = (float*)(W + p.ce0);
    }
    float* dgp = dgam ? (float*)(W + p.dgp) : nullptr;
    if (mem_fused(p.nb, gvec != nullptr)) {
      LAUNCH(ST_MEM_BWD, mem_bwd(dt, W + p.pbar, lo ? W + p.pbar_lo : nullptr, prm->Wm,
                                 (const float*)(SV + p.M), (float*)(W + p.dS), dgp,
                                 (float*)(W + p.dM), (float*)(W + p.mpart_b), p.B, p.nb, D,
                                 cfg->gamma, cr, s));
    } else {
      int nq = 0;
      LAUNCH(ST_WM_BWD, mem_bwd_proj(dt, W + p.pbar, lo ? W + p.pbar_lo : nullptr, prm->Wm,
                                     (float*)(W + p.mpart_b), p.B, p.nb, D, &nq, s));
      LAUNCH(ST_MEM_BWD, mem_bwd_scan(dt, (const float*)(SV + p.M), (float*)(W + p.dS), dgp,
                                      (float*)(W + p.mpart_b), nq, p.B, p.nb, D, cfg->gamma, cr,
                                      s));
    }
    if (chunk)
      LAUNCH(ST_CARRY_BWD, carry_finish((const float*)(SV + p.cN), (const float*)(SV + p.cZ),
                                        (const float*)(W + p.cdm), (const float*)(W + p.dS),
                                        (const float*)(W + p.ce0), dcin ? dcin->N : nullptr,
                                        dcin ? dcin->Z : nullptr,
                                        dgam ? (float*)(W + p.dgp) +
                                                   (size_t)dgr * (gvec ? D : 1)
                                             : nullptr,
                                        p.B, p.nb, D,
                                        cfg->gamma, gvec, gvec != nullptr, s));
    // Pooling backward: per-token a_t and ds_t, and partial sums of
    // ds_t H[t]; dwp = their sum on the side stream.
    LAUNCH(ST_POOL_BWD, pool_bwd(dt, SV + p.h, (const float*)(SV + p.s), (const float*)(SV + p.stats),
                                 (const float*)(SV + p.S), (const float*)(W + p.dS),
                                 (float*)(W + p.a), (float*)(W + p.ds),
                                 gr.dwp ? (float*)(W + p.dwpp) : nullptr, p.B, p.T, D, p.L, s));
    // (dwp, the sum of those partials, goes to the side stream with dWo.)
    // dH = dY + dU Wg^T + a_t dS[blk] + ds_t wp.
    {
      GemmDesc g{BT, D, D, W + p.du, D, false, {prm->Wg, nullptr, nullptr}, D, false, kSegNone, 0, 1};
      HbarEpi e{W + p.dh, dY, (const float*)(W + p.a), (const float*)(W + p.ds),
                (const float*)(W + p.dS), prm->wp, p.T, p.L, p.nb, D};
      LAUNCH(ST_HBAR, gemm_hbar(dt, g, e, s));
    }
  }  // the memory path's backward
  // Output projection backward: dHcat here, then dWo on the side stream,
  // where it overlaps the attention backward (a latency-bound kernel) rather
  // than competing with the dHcat product for the matrix cores.
  {
    GemmDesc g{BT, D, D, dH, D, false, {prm->Wo, nullptr, nullptr}, D, false, kSegNone, 0, 1};
    LAUNCH(ST_WO_DGRAD, gemm_store(dt, g, W + p.dout, D, false, nullptr, 0, s));
  }
  // dwp joins this branch rather than taking a fork of its own after the
  // pooling backward: each fork costs the caller's stream an event record.
  // So does the decay gradient's fixed-order sum of its partials.
  const bool dwp_side = gr.dwp && !single;
  const bool dg_side = dgam && !single;
  if (gr.dWo || dwp_side || dg_side) {
    SIDE_BEGIN();
    if (gr.dWo) {
      GemmDesc g{D, D, BT, SV + p.o, D, true, {dH, nullptr, nullptr}, D, true, kSegNone, 0, 1};
      LAUNCH_SPLITK(ST_WO_WGRAD, ST_WO_WGRAD_RED, dt, g, wpart, gr.dWo, nullptr, nullptr, D, D,
                    accum, dd_min_k(D, BT));
    }
    if (dwp_side)
      LAUNCH(ST_DWP, pool_dwp((float*)(W + p.dwpp), dt, p.B, p.T, D, p.L, gr.dwp, accum, s));
    if (dg_side)
      LAUNCH(ST_DGAMMA, dgamma_reduce((const float*)(W + p.dgp), dgr + (chunk ? p.B : 0),
                                      gvec ? D : 1, dgam, accum, s));
    SIDE_END();
  }
  // Block-local attention backward: one fused kernel when a block fits one
  // workgroup, else dQ (with delta) and then dK / dV.
  if (attn_bwd_fused(dt, p.T, D, p.H, p.L)) {
    LAUNCH(ST_ATTN_BWD_BLOCK,
           attn_bwd_block(dt, SV + p.qkv, SV + p.o, W + p.dout, (const float*)(SV + p.lse),
                          W + p.dqkv, p.B, p.T, D, p.H, p.L, s));
  } else {
    LAUNCH(ST_ATTN_BWD_DQ,
           attn_bwd_dq(dt, SV + p.qkv, SV + p.o, W + p.dout, (const float*)(SV + p.lse),
                       (float*)(W + p.delta), W + p.dqkv, p.B, p.T, D, p.H, p.L, s));
    LAUNCH(ST_ATTN_BWD_DKDV,
           attn_bwd_dkdv(dt, SV + p.qkv, W + p.dout, (const float*)(SV + p.lse),
                         (const float*)(W + p.delta), W + p.dqkv, p.B, p.T, D, p.H, p.L, s));
  }
  // Q/K/V projections backward: dW{q,k,v} on the side stream, dX here.
  if (gr.dWq || gr.dWk || gr.dWv) {
    SIDE_BEGIN();
    {
      GemmDesc g{D, 3 * D, BT, X, D, true, {W + p.dqkv, nullptr, nullptr}, 3 * D, true, kSegNone,
                 0, 1};
      LAUNCH_SPLITK(ST_QKV_WGRAD, ST_QKV_WGRAD_RED, dt, g, wpart, gr.dWq, gr.dWk, gr.dWv, D, D,
                    accum, kQkvMinK);
    }
    SIDE_END();
  }
  if (dX) {
    GemmDesc g{BT, D, 3 * D, W + p.dqkv, 3 * D, false, {prm->Wq, prm->Wk, prm->Wv}, D, false,
               kSegK, D, 1};
    LAUNCH(ST_DX, gemm_store(dt, g, dX, D, false, residual ? dY : nullptr, D, s));
  }
  // Join: later work on the caller's stream sees every side-stream result.
  if (nfork > 0 && order_after(main_s, side_s, ev_join) != hipSuccess) return BCMT_ERR_HIP;
#undef SIDE_BEGIN
#undef SIDE_END
  return BCMT_OK;
}

// ------------------------------------------------------------------ allocation-free forward
// The forward pass's workspace for bcmt_layer_forward_noalloc: one array per
// GPU, part of the loaded code object (each device holds its own copy until
// the process ends).  Host code never uses this name as an address: the
// device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[BCMT_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// The current device's copy of `scratch`, or null if it cannot be found.
void* scratch_for_current_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    g_scratch[dev] = ptr;
  }
  return g_scratch[dev];
}
}  // namespace

extern "C" {

int bcmt_layer_forward(const bcmt_config* cfg, const void* X, const bcmt_params* prm, void* Y,
                       void* saved, void* ws, size_t ws_bytes, void* stream) {
  return layer_forward(cfg, X, prm, Y, saved, ws, ws_bytes, stream, false, nullptr, nullptr);
}

int bcmt_layer_forward_noalloc(const bcmt_config* cfg, const void* X, const bcmt_params* prm,
                               void* Y, void* saved, void* stream) {
  // Every check that needs no device comes first, so that a size beyond the
  // scratch array is rejected before any HIP call.
  const int st = check_config(cfg);
  if (st != BCMT_OK) return st;
  if (!saved) return BCMT_ERR_INVALID;
  if (Plan(*cfg).fwd_bytes > (size_t)BCMT_NOALLOC_SCRATCH_BYTES) return BCMT_ERR_WORKSPACE;
  void* ws = scratch_for_current_device();
  if (!ws) return BCMT_ERR_HIP;
  return layer_forward(cfg, X, prm, Y, saved, ws, (size_t)BCMT_NOALLOC_SCRATCH_BYTES, stream,
                       false, nullptr, nullptr);
}

int bcmt_layer_backward(const bcmt_config* cfg, const void* X, const bcmt_params* prm,
                        const void* saved, const void* dY, void* dX, const bcmt_grads* grads,
                        void* ws, size_t ws_bytes, void* stream, const bcmt_side* side) {
  return layer_backward(cfg, X, prm, saved, dY, dX, grads, ws, ws_bytes, stream, side, false,
                        nullptr, nullptr);
}

int bcmt_layer_forward_chunk(const bcmt_config* cfg, const void* X, const bcmt_params* prm,
                             const bcmt_carry* carry_in, void* Y, const bcmt_carry* carry_out,
                             void* saved, void* ws, size_t ws_bytes, void* stream) {
  return layer_forward(cfg, X, prm, Y, saved, ws, ws_bytes, stream, true, carry_in, carry_out);
}

int bcmt_layer_backward_chunk(const bcmt_config* cfg, const void* X, const bcmt_params* prm,
                              const void* saved, const void* dY, const bcmt_carry* dcarry_out,
                              void* dX, const bcmt_carry* dcarry_in, const bcmt_grads* grads,
                              void* ws, size_t ws_bytes, void* stream,
                              const bcmt_side* side) {
  return layer_backward(cfg, X, prm, saved, dY, dX, grads, ws, ws_bytes, stream, side, true,
                        dcarry_out, dcarry_in);
}

size_t bcmt_decode_state_bytes(const bcmt_config* cfg) {
  if (check_decode(cfg) != BCMT_OK) return 0;
  return DecPlan(*cfg).state_bytes;
}

size_t bcmt_decode_workspace_bytes(const bcmt_config* cfg) {
  if (check_decode(cfg) != BCMT_OK) return 0;
  return DecPlan(*cfg).ws_bytes;
}

int bcmt_decode_reset(const bcmt_config* cfg, const bcmt_params* prm, const bcmt_carry* carry_in,
                      void* state, void* ws, size_t ws_bytes, void* stream) {
  int st = check_decode(cfg);
  if (st != BCMT_OK) return st;
  if (!prm || !prm->Wm || !aligned16(prm->Wm) || !carry_ok(carry_in) || !decay_ok(cfg, prm))
    return BCMT_ERR_INVALID;
  if (!state || !aligned16(state) || !ws || !aligned16(ws)) return BCMT_ERR_INVALID;
  DecPlan p(*cfg);
  if (ws_bytes < p.ws_bytes) return BCMT_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  char* S = (char*)state;
  char* W = (char*)ws;
  // The memory state and the first block's context (N / Z) Wm, or zeros.
  LAUNCH(ST_DEC_RESET, carry_prep(p.dt, carry_in ? carry_in->N : nullptr,
                                  carry_in ? carry_in->Z : nullptr, (float*)(S + p.N),
                                  (float*)(S + p.Z), W + p.Mt,
                                  carry_in ? nullptr : (float*)(S + p.C), p.B, p.D,
                                  channel_decay(cfg, prm) != nullptr, s));
  if (carry_in)
    LAUNCH(ST_DEC_RESET, carry_proj(p.dt, W + p.Mt, prm->Wm, (float*)(S + p.C),
                                    (float*)(W + p.cpart), false, false, p.B, p.D, s));
  return BCMT_OK;
}

int bcmt_decode_step(const bcmt_config* cfg, const bcmt_params* prm, int64_t t, const void* x,
                     void* y, void* state, void* ws, size_t ws_bytes, void* stream) {
  int st = check_decode(cfg);
  if (st != BCMT_OK) return st;
  if (t < 0 || !x || !y || !prm || !state || !ws || !decay_ok(cfg, prm)) return BCMT_ERR_INVALID;
  const void* w[7] = {prm->Wq, prm->Wk, prm->Wv, prm->Wo, prm->Wm, prm->Wg, prm->wp};
  for (const void* q : w)
    if (!q || !aligned16(q)) return BCMT_ERR_INVALID;
  if (!aligned16(x) || !aligned16(y) || !aligned16(state) || !aligned16(ws))
    return BCMT_ERR_INVALID;
  DecPlan p(*cfg);
  if (overlaps(x, y, (size_t)p.B * p.D * p.es)) return BCMT_ERR_INVALID;
  if (ws_bytes < p.ws_bytes) return BCMT_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  char* S = (char*)state;
  char* W = (char*)ws;
  const int off = (int)(t % p.L);
  float* part = (float*)(W + p.part);
  const int D = p.D;
  const int ks3 = dec_splits(p.dt, D, 3 * D, p.B), ks1 = dec_splits(p.dt, D, D, p.B);
  // [q k v] = x [Wq Wk Wv] (K-split partial sums), then attention over the
  // block's cache, which first adds them up and appends k and v.
  LAUNCH(ST_DEC_QKV, dec_product(p.dt, x, D, prm->Wq, prm->Wk, prm->Wv, p.B, D, 3 * D, part, s));
  LAUNCH(ST_DEC_ATTN, dec_attn(p.dt, part, ks3, S + p.Kc, S + p.Vc, W + p.o, p.B, D, p.H, p.L,
                               off, s));
  // h = o Wo (cached, with its pooling score), then the gate and injection.
  LAUNCH(ST_DEC_WO, dec_product(p.dt, W + p.o, D, prm->Wo, nullptr, nullptr, p.B, D, D, part, s));
  LAUNCH(ST_DEC_WO_FIN, dec_wo_finish(p.dt, part, ks1, prm->wp, S + p.Hc, (float*)(S + p.spc),
                                      p.B, D, p.L, off, s));
  char* hrow = S + p.Hc + (size_t)off * D * p.es;
  LAUNCH(ST_DEC_GATE, dec_product(p.dt, hrow, (int64_t)p.L * D, prm->Wg, nullptr, nullptr, p.B, D,
                                  D, part, s));
  LAUNCH(ST_DEC_GATE_FIN, dec_gate_finish(p.dt, part, ks1, S + p.Hc, (const float*)(S + p.C),
                                          (cfg->flags & BCMT_FLAG_RESIDUAL) ? x : nullptr, y, p.B,
                                          D, p.L, off, s));
  if (off == p.L - 1) {
    // The block is complete: its summary enters the memory, which gives the
    // next block's context.
    LAUNCH(ST_DEC_POOL, dec_pool(p.dt, S + p.Hc, (const float*)(S + p.spc), (float*)(S + p.N),
                                 (const float*)(S + p.Z), W + p.Mt, p.B, D, p.L, cfg->gamma,
                                 channel_decay(cfg, prm), s));
    LAUNCH(ST_DEC_MEM, dec_product(p.dt, W + p.Mt, D, prm->Wm, nullptr, nullptr, p.B, D, D, part,
                                   s));
    LAUNCH(ST_DEC_MEM_FIN, dec_mem_finish(part, ks1, (float*)(S + p.C), (float*)(S + p.Z), p.B, D,
                                          cfg->gamma, channel_decay(cfg, prm), s));
  }
  return BCMT_OK;
}

}  // extern "C"
