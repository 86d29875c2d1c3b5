// Host-side launchers of the BCMT kernels (internal to the library).
// Every launcher enqueues on the given stream and returns the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bcmt {

enum class DType { F32 = 0, BF16 = 1 };

// ------------------------------------------------------------------ GEMM
// C[m, n] = sum_k A(m, k) * B(k, n), float32 accumulation.
//   A(m, k) = A[m * lda + k]            (a_mcontig = false)
//           = A[k * lda + m]            (a_mcontig = true)
//   B(k, n) = Bseg[n * ldb + k]         (b_ncontig = false)
//           = Bseg[k * ldb + n]         (b_ncontig = true)
// B may be split into up to three pointers along N (seg = kSegN) or along K
// (seg = kSegK), each covering seg_len indices; the index inside a pointer is
// the global index minus seg * seg_len.
// Contiguous dimensions (K when an operand is K-contiguous, M or N
// otherwise) must be multiples of 8 elements.
enum { kSegNone = 0, kSegN = 1, kSegK = 2 };

struct GemmDesc {
  int M, N, K;
  const void* A;
  int64_t lda;
  bool a_mcontig;
  const void* B[3];
  int64_t ldb;
  bool b_ncontig;
  int seg;
  int seg_len;
  int splits;  // split-K factor
  int kchunk;  // if > 0: K range per split (a multiple of 64), overriding splits
};

// Plain store: C = acc (+ add), C in the compute type or float32.
hipError_t gemm_store(DType dt, const GemmDesc& g, void* C, int64_t ldc, bool c_f32,
                      const void* add, int64_t ld_add, hipStream_t s);

// Weight-gradient product (large K): split-K partial tiles written to
// `partial` (float32), then a reduction over the splits that writes, or
// with `accumulate` adds into, up to three outputs split along N (a null
// output is skipped).  The split count is chosen here; g.splits is ignored.
// Deterministic: no atomics.
size_t gemm_wgrad_partial_bytes(int M, int N, int K);
// General split-K product into float32 outputs (any layout without B
// segments), every split at least min_k deep; with a single split the
// outputs are written directly and `partial` is unused.
size_t gemm_splitk_partial_bytes(int M, int N, int K, int min_k);
// The number of splits gemm_splitk chooses for that product.
int gemm_splitk_splits(int M, int N, int K, int min_k);
hipError_t gemm_splitk(DType dt, const GemmDesc& g, float* partial, float* C0, float* C1,
                       float* C2, int64_t ldc, int seg_len_n, bool accumulate, int min_k,
                       hipStream_t s);
// The two launches of gemm_splitk separately: the product (which writes the
// outputs itself when the plan has one split) and, when *splits > 1, the
// reduction of the partial tiles.
hipError_t gemm_splitk_product(DType dt, const GemmDesc& g, float* partial, float* C0, float* C1,
                               float* C2, int64_t ldc, int seg_len_n, bool accumulate, int min_k,
                               int* splits, hipStream_t s);
hipError_t gemm_splitk_reduce(const float* partial, int splits, int M, int N, float* C0, float* C1,
                              float* C2, int64_t ldc, int seg_len_n, bool accumulate,
                              hipStream_t s);
hipError_t gemm_wgrad(DType dt, const GemmDesc& g, float* partial, float* C0, float* C1,
                      float* C2, int64_t ldc, int seg_len_n, bool accumulate, hipStream_t s);

// Output projection with the pooling scores: C = acc ([M, N], row stride N)
// and sp[m * (N / 64) + q] = sum over columns 64q .. 64q+63 of C[m, n] wp[n]
// (N a multiple of 64; A K-contiguous, B N-contiguous).
hipError_t gemm_score(DType dt, const GemmDesc& g, void* C, const void* wp, float* sp,
                      hipStream_t s);

// Gate + injection epilogue (forward): U = acc;
//   G = sigmoid(U); Y = H + G * Mc[blk(t)] (+ X); G is stored for backward.
// Mc[b, i] = P[b, i - 1] for i >= 1 and 0 for i = 0 (the one-block shift).
// A chunk that follows earlier blocks (Pc not null) gives its block 0
// Mc = Pc[b] instead.
struct GateEpi {
  void* Y;
  void* G;
  const void* H;
  const void* X;     // nullable: residual off
  const float* P;    // [B * nb, D] projected memory
  int T, L, nb, D;
  const float* Pc;   // nullable: [B, D] projected memory of the earlier blocks
};
hipError_t gemm_gate(DType dt, const GemmDesc& g, const GateEpi& e, hipStream_t s);

// Backward of the local representation: dH = acc + dY + a_t * dS[blk] + ds_t * wp.
struct HbarEpi {
  void* dH;
  const void* dY;
  const float* a;     // [B*T] pooling weights
  const float* ds;    // [B*T] pooling-score gradients
  const float* dS;    // [B * nb, D] summary gradients
  const void* wp;     // [D]
  int T, L, nb, D;
};
hipError_t gemm_hbar(DType dt, const GemmDesc& g, const HbarEpi& e, hipStream_t s);

// Language-model MLP (bf16 only; A K-contiguous): U = acc and A = gelu(U)
// (tanh form, of the rounded U), both [M, N] with row stride ld; and the
// backward dU = acc * gelu'(U) with U as stored by gemm_gelu.
hipError_t gemm_gelu(DType dt, const GemmDesc& g, void* U, void* A, int64_t ld, hipStream_t s);
hipError_t gemm_gelu_bwd(DType dt, const GemmDesc& g, const void* U, void* dU, int64_t ld,
                         hipStream_t s);
// The tied head (bf16, A = f K-contiguous, B = E with B[k][v] = E[v][k],
// M >= 8, K a multiple of 64, N = the vocabulary padded to a multiple of
// 128): gemm_head_stats writes per row and 128-column tile (max, sum of
// exp(z - max)) over the columns below V to part (float pairs, row-major
// [M][N / 128]); gemm_head_grad writes G[m][n] = (softmax(z)[n] - [n ==
// tgt[m]]) * inv_n as bf16, zero for n >= V, given lse[m].
hipError_t gemm_head_stats(const GemmDesc& g, float* part, int V, hipStream_t s);
hipError_t gemm_head_grad(const GemmDesc& g, void* G, int64_t ld, const float* lse,
                          const int32_t* tgt, int V, float inv_n, hipStream_t s);
// The same two passes without a tiled product, for d = 128 (head.hip): each
// workgroup streams a range of the vocabulary past 128 rows of f held in
// registers.  head_stats writes *nrange (max, sum of exp(z - max)) pairs
// per row to part (row-major [rows][*nrange], natural units), for the
// log-sum-exp kernel; head_grad writes G as gemm_head_grad does and df =
// G E (float32 [rows][128]), through dfpart (head_partial_bytes) when the
// vocabulary is split into several ranges.
bool head_fused_ok(int d, int Vp);
size_t head_partial_bytes(int rows, int d, int Vp);
hipError_t head_stats(const void* f, const void* E, int rows, int d, int V, int Vp, float* part,
                      int* nrange, hipStream_t s);
hipError_t head_grad(const void* f, const void* E, int rows, int d, int V, int Vp,
                     const float* lse, const int32_t* tgt, float inv_n, void* G, int64_t ldg,
                     float* dfpart, float* df, hipStream_t s);

// ------------------------------------------------------------------ attention
// qkv: [B, T, 3D] (Q | K | V), head h at columns h*64 .. h*64+63 of each.
hipError_t attn_fwd(DType dt, const void* qkv, void* out, float* lse, int B, int T, int D,
                    int H, int L, hipStream_t s);
// Backward in two passes: dQ (also writes delta_t = dO_t . O_t), then dK/dV.
hipError_t attn_bwd_dq(DType dt, const void* qkv, const void* out, const void* dout,
                       const float* lse, float* delta, void* dqkv, int B, int T, int D, int H,
                       int L, hipStream_t s);
hipError_t attn_bwd_dkdv(DType dt, const void* qkv, const void* dout, const float* lse,
                         const float* delta, void* dqkv, int B, int T, int D, int H, int L,
                         hipStream_t s);
// Whether attn_bwd_block serves this layer (bf16, blocks of at most 128
// tokens), and the fused backward of each block in one workgroup (dQ, dK,
// dV; delta is formed internally and not written).
bool attn_bwd_fused(DType dt, int T, int D, int H, int L);
hipError_t attn_bwd_block(DType dt, const void* qkv, const void* out, const void* dout,
                          const float* lse, void* dqkv, int B, int T, int D, int H, int L,
                          hipStream_t s);

// Heads of 16 or 32 dimensions (attention_small.hip): the same three
// passes (forward, dQ with delta, dK / dV) in float32 vector arithmetic;
// attn_fwd / attn_bwd_dq / attn_bwd_dkdv route such layers there.
bool attn_small_heads(int D, int H);
hipError_t attn_small_fwd(DType dt, const void* qkv, void* out, float* lse, int B, int T, int D,
                          int H, int L, hipStream_t s);
hipError_t attn_small_dq(DType dt, const void* qkv, const void* o, const void* dout,
                         const float* lse, float* delta, void* dqkv, int B, int T, int D, int H,
                         int L, hipStream_t s);
hipError_t attn_small_dkdv(DType dt, const void* qkv, const void* dout, const float* lse,
                           const float* delta, void* dqkv, int B, int T, int D, int H, int L,
                           hipStream_t s);

// ------------------------------------------------------------------ memory path
// State of the decayed memory recurrence shared by consecutive chunks of the
// same sequences (float32).  Forward: N and Z before the chunk's first block
// (Nin [B, D], Zin [B]; null: empty history), Pc = (Nin / Zin) Wm [B, D]
// (read by the fused scan), and where to write N and Z after the last block
// (Nout, Zout; nullable).  Backward: the gradients arriving for that final
// state (dNout, dZout; nullable) and the per-column gradient of Z at the
// first block (e0 [B, D]; nullable).  All members null: a whole sequence.
// With a per-channel decay (gvec [D], not null) every channel has its own
// normaliser: Zin, Zout and dZout are then [B, D] (zcol), the scalar gamma
// argument is unused, and the backward adds the decay gradient per channel
// into dgamma [D] instead of into one scalar.
struct Carry {
  const float* Nin = nullptr;
  const float* Zin = nullptr;
  const float* Pc = nullptr;
  float* Nout = nullptr;
  float* Zout = nullptr;
  const float* dNout = nullptr;
  const float* dZout = nullptr;
  float* e0 = nullptr;
  const float* gvec = nullptr;
  bool zcol = false;
};
// Pooling, from the np partial scores per token written by gemm_score:
// scores s [B*T], summaries S [B*nb, D] (float32, and St in the compute
// type) and per-block softmax statistics (max, normaliser) [B*nb, 2].
// Also clears zero[0 .. nzero) (may be null), shared among its workgroups.
hipError_t pool_fwd(DType dt, const void* H, const float* sp, int np, float* s_out, float* S,
                    void* St, float* stats, int B, int T, int D, int L, float* zero,
                    int64_t nzero, hipStream_t s);
// Memory forward: M (float32), Mt (compute type) and P = M Wm from S.  Up
// to a few dozen blocks per sequence one kernel does it all (Q = St Wm with
// St = S in the compute type, [B*nb, D], and the decayed scans of S and Q);
// for longer sequences Q is a split-K product whose partials a parallel
// scan of S and Q adds up, using `part` (mem_part_bytes bytes; may be null
// when that is 0).
// The single kernel scans the projected summaries, which equals projecting
// the scan only for one decay shared by the channels: a per-channel decay
// takes the scan + matrix-product path at any length.
bool mem_fused(int nb, bool per_channel);
size_t mem_part_bytes(int B, int nb, int D, bool per_channel);
// The look-back scans' records inside `part` (null and *nfloat = 0 where a
// call with these sizes does not use them): a kernel earlier on the stream
// must clear these *nfloat floats (pool_fwd's `zero` before the forward,
// gate_bwd's zero_a before the backward).
float* mem_lb_flags(float* part, int B, int nb, int D, bool per_channel, bool carry,
                    int64_t* nfloat);
hipError_t mem_fwd(DType dt, const void* St, const void* Wm, const float* S, float* M, void* Mt,
                   float* P, float* part, int B, int nb, int D, float gamma, const Carry& c,
                   hipStream_t s);
// The long path's steps (what mem_fwd / mem_bwd run when mem_fused is
// false), for callers that time them apart: mem_fwd_proj is the W_m
// product (one decay: Q = St Wm as *nq split-K slices, before the scan; per
// channel: P = Mt Wm, after it), mem_fwd_scan the two scan passes;
// mem_bwd_proj the product dM = [hi | lo] [Wm^T; Wm^T] (*nq slices),
// mem_bwd_scan the reverse scans.
hipError_t mem_fwd_proj(DType dt, const void* St, const void* Wm, const void* Mt, float* P,
                        float* part, int B, int nb, int D, bool per_channel, int* nq,
                        hipStream_t s);
hipError_t mem_fwd_scan(DType dt, const float* S, float* M, void* Mt, float* P, float* part, int nq,
                        int B, int nb, int D, float gamma, const Carry& c, hipStream_t s);
hipError_t mem_bwd_proj(DType dt, const void* Pbar, const void* Pbar_lo, const void* Wm,
                        float* part, int B, int nb, int D, int* nq, hipStream_t s);
hipError_t mem_bwd_scan(DType dt, const float* M, float* dS, float* dgpart, float* part, int nq,
                        int B, int nb, int D, float gamma, const Carry& c, hipStream_t s);
// Gate backward; also zeroes zero_a[0..na) and *zero_b (either may be null).
// With Pc (a chunk after earlier blocks) block 0 uses Mc = Pc[b] and its
// sum of dY * G goes to Pbar_c [B, D] (compute type).  In bf16, with
// Pbar_lo not null, each block sum v is kept as hi = bf16(v) and lo =
// bf16(v - hi) in one row [hi (D) | lo (D)] of Pbar (rows 2D apart; Pbar_lo
// marks that layout and is Pbar + D), and Pbar_c_lo holds the lo part of
// Pbar_c; float32 ignores them.
hipError_t gate_bwd(DType dt, const void* dY, const void* G, const float* P, void* dU,
                    void* Pbar, void* Pbar_lo, float* zero_a, int na, float* zero_b, int B, int T,
                    int D, int L, const float* Pc, void* Pbar_c, void* Pbar_c_lo, hipStream_t s);
// Memory backward: dM = (hi + lo) Wm^T over the rows of Pbar (the layout
// gate_bwd writes; Pbar_lo null: rows of D values, hi alone; float32
// ignores it), then the reverse decayed scan: dS and the decay gradient as
// partials (when dgpart is given): dg_part_rows(B, nb, D, per channel) rows
// of 1 float (one decay) or D floats (one per channel), every row written.
// For long sequences (see mem_fwd) dM goes through a split-K product using
// `part`; both may be null for short ones.
hipError_t mem_bwd(DType dt, const void* Pbar, const void* Pbar_lo, const void* Wm,
                   const float* M, float* dS, float* dgpart, float* dM, float* part, int B, int nb,
                   int D, float gamma, const Carry& c, hipStream_t s);
int dg_part_rows(int B, int nb, int D, bool per_channel);
// The rows one call writes: without carried state (carry false) and few
// sequences, the long path's look-back scans write one row per (sequence,
// column slice, segment); dg_part_rows is the most over both kinds of call.
int dg_part_rows_used(int B, int nb, int D, bool per_channel, bool carry);
// out[0 .. Dp) = (out if accumulate, else 0) + the sum of part[rows][Dp]
// over its rows, in a fixed order (deterministic).
hipError_t dgamma_reduce(const float* part, int rows, int Dp, float* out, bool accumulate,
                         hipStream_t s);
// Chunked execution.  carry_prep copies the incoming state (Nu [B, D],
// Zu [B]; both null: empty history) to Nin / Zin and writes its memory
// Mct = Nin / Zin (0 where Zin = 0) in the compute type; with no incoming
// state it also zeroes Pc.  carry_proj: Pc = Mct Wm, or with `transposed`
// dMc = Pbar_c Wm^T, both [B, D] float32 (added into `out` with
// `accumulate`), using `part`
// (carry_part_bytes bytes).  carry_finish forms the incoming state's
// gradients from dMc, dS of block 0 and e0:
//   dNin = dMc / Zin + g dS_0,  dZin = sum_cols (g e0 - dMc . M_in / Zin),
// and writes the first block's decay term sum_cols dS_0 Nin + e0 Zin as
// B more partial rows at dgpart (1 or D floats each, as mem_bwd's); null
// outputs are skipped.
hipError_t carry_prep(DType dt, const float* Nu, const float* Zu, float* Nin, float* Zin,
                      void* Mct, float* Pc, int B, int D, bool zcol, hipStream_t s);
size_t carry_part_bytes(int B, int D);
hipError_t carry_proj(DType dt, const void* A, const void* Wm, float* out, float* part,
                      bool transposed, bool accumulate, int B, int D, hipStream_t s);
hipError_t carry_finish(const float* Nin, const float* Zin, const float* dMc, const float* dS,
                        const float* e0, float* dNin, float* dZin, float* dgpart, int B, int nb,
                        int D, float gamma, const float* gvec, bool zcol, hipStream_t s);
// Pooling backward: per-token softmax weights a_t and score gradients ds_t,
// and (when dwp_part is not null) partial sums of ds_t H[t] over chunks of
// tokens, one row of D floats per chunk.
hipError_t pool_bwd(DType dt, const void* H, const float* s_in, const float* stats,
                    const float* S, const float* dS, float* a_out, float* ds_out,
                    float* dwp_part, int B, int T, int D, int L, hipStream_t s);
// Rows of D floats the dwp_part workspace needs (partial sums and the
// reduction's intermediate rows).
int64_t pool_bwd_partial_rows(DType dt, int B, int T, int D, int L);
// dwp = (or +=) the sum of the partial rows, in a fixed order.
hipError_t pool_dwp(float* dwp_part, DType dt, int B, int T, int D, int L, float* dwp,
                    bool accumulate, hipStream_t s);
hipError_t fill_f32(float* p, int64_t n, float v, hipStream_t s);

// ------------------------------------------------------------------ decoding
// One more token per sequence (decode.hip).  The block caches hold, per
// sequence, L rows of D: keys Kc, values Vc and local outputs Hc (compute
// type), and the score parts spc [B, L, D / 64] (float32); N, Z and C are
// the memory state and the current block's context (float32).  `off` is
// the new token's slot in its block.  A product x [B, D] (row stride ldx)
// times [D, N] (W0 | W1 | W2, D columns each, or W0 alone with N = D)
// writes dec_splits() K-split partial sums to `part` (dec_part_bytes), which
// the next kernel adds up.
int dec_max_blocklen();
int dec_max_batch();
int dec_score_parts(int D);
int dec_splits(DType dt, int K, int N, int B);
size_t dec_part_bytes(DType dt, int B, int D);
hipError_t dec_product(DType dt, const void* x, int64_t ldx, const void* W0, const void* W1,
                       const void* W2, int B, int D, int N, float* part, hipStream_t s);
// Adds the QKV splits (k and v to the caches at off), then attention -> o.
hipError_t dec_attn(DType dt, const float* part, int ks, void* Kc, void* Vc, void* o, int B, int D,
                    int H, int L, int off, hipStream_t s);
// h = sum of the splits -> Hc at off, with its score parts -> spc.
hipError_t dec_wo_finish(DType dt, const float* part, int ks, const void* wp, void* Hc, float* spc,
                         int B, int D, int L, int off, hipStream_t s);
// y = h + sigmoid(u) C (+ x), u = sum of the splits.
hipError_t dec_gate_finish(DType dt, const float* part, int ks, const void* Hc, const float* C,
                           const void* x, void* y, int B, int D, int L, int off, hipStream_t s);
// After the block's last token: pooling, N = g N + S, Mt = N / (g Z + 1).
// With a per-channel decay gvec [D], g and Z are per channel (Z [B, D]).
hipError_t dec_pool(DType dt, const void* Hc, const float* spc, float* N, const float* Z, void* Mt,
                    int B, int D, int L, float gamma, const float* gvec, hipStream_t s);
// C = sum of the splits of Mt Wm, Z = g Z + 1.
hipError_t dec_mem_finish(const float* part, int ks, float* C, float* Z, int B, int D, float gamma,
                          const float* gvec, hipStream_t s);

}  // namespace bcmt
