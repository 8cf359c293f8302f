// Host-side launchers of the device kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dllm_rps.h"

#define DLLM_TOPK_REG 16  // top-K entries kept per row in registers

namespace dllm {

struct QkvOut {
  void* q;           // [B][H][seq][hd]
  void* k;           // [B][H][seq][hd]
  void* vt;          // [B][H][hd][vt_ld]
  int seq, vt_ld, pos_offset, H, hd, d;
  const float2* rope;  // [max_pos][hd/2] (cos, sin)
  // packed lookahead (see AttnArgs): row r >= pack_S has the position of row
  // pack_b0 + (r - pack_S) % pack_B (pack_B a power of two); pack_B == 0: row
  // r has pos_offset + r
  int pack_S = 0, pack_b0 = 0, pack_B = 0;
};

// Split-K of a projection GEMM with few rows: `splits` parts of the K range
// write fp32 partial tiles to `part` (gemm_partial_bytes), reduced in a fixed
// order by a second kernel that applies the epilogue.  splits <= 1: one pass.
struct SplitK {
  float* part;
  int splits;
  bool defer = false;   // resid: write the partials only; the caller adds them (resid_rmsnorm / splitk_add)
};
// split-K parts of a projection of M rows, N outputs (gate/up: 2 F, the
// gate and up rows) and depth K
enum { GEMM_KIND_QKV = 0, GEMM_KIND_RESID = 1, GEMM_KIND_GATEUP = 2 };
int gemm_splits(int kind, int M, int N, int K, int dtype);
size_t gemm_partial_bytes(int M, int tiles_n, int splits);

// X[M][N] (fp32, row stride ldx) += A[M][K] B[N][K]^T
hipError_t gemm_resid(int dtype, const void* A, int lda, const void* B, int ldb, int M, int N, int K, float* X,
                      int ldx, hipStream_t s, const SplitK* sk = nullptr);
// out[M][F] = silu(A Wg^T) * (A Wu^T) with Wgu = [Wg; Wu] ([2F][K])
hipError_t gemm_swiglu(int dtype, const void* A, int lda, const void* Wgu, int M, int F, int K, void* out,
                       hipStream_t s, const SplitK* sk = nullptr);
// Q/K/V projection with rotary embedding on Q and K, scattered head-major
hipError_t gemm_qkv(int dtype, const void* A, int lda, const void* Wqkv, int M, int K, const QkvOut& o,
                    hipStream_t s, const SplitK* sk = nullptr);

// x[M][N] += the deferred split-K partials of gemm_resid (fixed order)
hipError_t splitk_add(const SplitK& sk, int M, int N, float* X, int ldx, hipStream_t s);
// x[r] += the deferred split-K partials of gemm_resid (row pitch np), then
// out[r] = rmsnorm(x[r]), for rows 0 .. M-1
hipError_t resid_rmsnorm(int dtype, const float* part, int splits, int np, int M, float* x, int d, float eps,
                         void* out, hipStream_t s);

// x[r][:] = emb[tok[r]][:] as fp32
hipError_t embed(int dtype, const int32_t* tok, int rows, const void* emb, int d, int vocab, float* x, hipStream_t s);
// out[r] = x[src(r)] / sqrt(mean(x^2) + eps); src(r) = r, or b * seq + pos[j] for
// r = b * n_pos + j when pos is given
hipError_t rmsnorm(int dtype, const float* x, int d, float eps, int rows, const int32_t* pos, int n_pos, int seq,
                   void* out, hipStream_t s);

struct AttnArgs {
  const void* q;     // [B][H][Sq][hd]
  const void* k;     // [B][H][Sq][hd]
  const void* vt;    // [B][H][hd][vt_ld]
  int B, H, Sq, hd, vt_ld;
  const void* kp;    // nullable prefix keys [H][cap][hd]
  const void* vpt;   // prefix values^T [H][hd][cap]
  int p_len, p_cap;
  void* o;           // [B*Sq][H*hd]
  // packed lookahead (B == 1): rows 0 .. pack_S-1 are the shared sequence,
  // then branch blocks of pack_B rows, each standing in for rows
  // pack_b0 .. pack_b0+pack_B-1; a cached prefix stays visible to every row;
  // pack_B == 0: no packing
  int pack_S = 0, pack_b0 = 0, pack_B = 0;
  // split layout with few workgroups: the keys are split over workgroups whose
  // partial softmax states are merged afterwards; workspace of
  // attn_partial_bytes (nullable: no key split)
  float* kv_part = nullptr;
};
hipError_t attention(int dtype, const AttnArgs& a, hipStream_t s);
// workspace for the key split of an attention over B x H x Sq queries (0: never split)
size_t attn_partial_bytes(int B, int H, int Sq, int hd);

// LM-head rows of a packed lookahead forward: (1 + n_branch) * n_lm rows, the
// shared sequence's then each branch's; row[] is the packed row each reads,
// src[] its in-sequence position (the row-scale index)
hipError_t packed_lm_rows(int S, int b0, int B, int n_branch, const int32_t* lm_pos, int n_lm, int32_t* row,
                          int32_t* src, hipStream_t s);

// copy this call's K and V^T (batch 1) into a cache at positions off .. off+seq-1
hipError_t kv_store(int dtype, const void* k, const void* vt, int H, int seq, int hd, int vt_ld, void* ck,
                    void* cvt, int cap, int off, hipStream_t s);

struct StatsOut {
  float* H;
  float* lse;
  float* lmax;
  int32_t* argmax;
  int32_t* topk_id;
  float* topk_logit;
  int k;
};
size_t lmhead_workspace(int R, int V);
// Pass 1 writes per-slice partial statistics to ws; pass 2 merges them into out.
// row_scale (nullable) is indexed by rs_idx[row % rs_n] clamped to [0, rs_lim) (or row % rs_n without rs_idx)
hipError_t lmhead_partials(int dtype, const void* h, const void* w, int R, int d, int V, const float* row_scale,
                           const int32_t* rs_idx, int rs_n, int rs_lim, float scale, int mask_id, void* ws,
                           hipStream_t s);
hipError_t lmhead_merge(int R, int V, const StatsOut& out, void* ws, hipStream_t s);
hipError_t probe_logits(int dtype, const void* h, const void* w, int d, int V, int R, const int32_t* row,
                        const int32_t* tok, int n, const float* row_scale, const int32_t* rs_idx, int n_pos,
                        int rs_lim, float scale, float* out, hipStream_t s);

// scheduler (single-workgroup kernels)
hipError_t rps_select(const StatsOut& base, const int32_t* m_pos, int n_m, const rps_params& prm, rps_plan* plan,
                      hipStream_t s);
hipError_t rps_branches(const int32_t* tokens, int seq, const rps_plan* plan, int anchor_first, int capacity,
                        int32_t* out, hipStream_t s);
// packed lookahead tokens: out[seq + capacity * B] = tokens, then one copy of
// the block b0 .. b0+B-1 per branch slot with that branch's pivot filled
hipError_t rps_branches_packed(const int32_t* tokens, int seq, const rps_plan* plan, int b0, int B, int capacity,
                               int32_t* out, hipStream_t s);
hipError_t rps_score(const StatsOut& anchor, const StatsOut& branches, int branch_offset, int n_m,
                     const rps_plan* plan, const float* anchor_logit, float lambda, float* scores, float* deltas,
                     rps_decision* dec, hipStream_t s);
hipError_t rps_commit_step(int32_t* tokens, int seq, int32_t* m_pos, int n_m, const StatsOut& base, const rps_decision* dec,
                           const StatsOut* branches, int branch_offset, const StatsOut* anchor, float tau,
                           int32_t* n_m_out, int32_t* committed, int32_t* n_committed, hipStream_t s);
hipError_t sched_commit_step(int32_t* tokens, int seq, int32_t* m_pos, int n_m, const StatsOut& st, int rule, int k,
                            int32_t* n_m_out, int32_t* committed, int32_t* n_committed, hipStream_t s);

// register-only bf16 MFMA loop (benchmark calibration); *flop: the launch's MFMA work
hipError_t mfma_calibration(bool random_operands, int iters, int workgroups, double* flop, hipStream_t s);

}  // namespace dllm
