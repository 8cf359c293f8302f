// Scheduler kernels of one RPS step (Section 4.1, Algorithm 1): pivot
// selection and candidate sets, lookahead batch construction, Eq. 4 scoring
// with the commit/abstain decision, and the commit / carry-over / compaction
// of the masked set.  Each runs as a single workgroup over at most
// RPS_MAX_MASKED masked positions; they are latency-bound and carry every
// integer decision of the step.
#include "dllm_rps.h"
#include "kernels.h"
#include "common.h"

namespace dllm {

namespace {

constexpr int kT = 256;
constexpr int kMaxM = RPS_MAX_MASKED;

struct StatsIn {
  const float* H;
  const float* lse;
  const float* lmax;
  const int32_t* argmax;
  const int32_t* topk_id;
  const float* topk_logit;
  int k;
};

// block-wide (value, id) argmax over 256 threads; result valid in every thread
__device__ void block_argmax(float& v, int& i, float* sv, int* si) {
  wave_argmax(v, i);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) { sv[w] = v; si[w] = i; }
  __syncthreads();
  v = sv[0];
  i = si[0];
  for (int k = 1; k < kT / kWave; ++k)
    if (better(sv[k], si[k], v, i)) { v = sv[k]; i = si[k]; }
  __syncthreads();
}

__global__ __launch_bounds__(kT) void select_kernel(StatsIn st, const int32_t* __restrict__ m_pos, int n_m,
                                                    rps_params prm, rps_plan* __restrict__ plan) {
  __shared__ float sh_sort[kMaxM];
  __shared__ float sh_htr[kMaxM];
  __shared__ uint8_t sh_feas[kMaxM];
  __shared__ float red_v[4];
  __shared__ int red_i[4];
  __shared__ int chosen[RPS_MAX_PIVOTS];
  __shared__ float band[2];
  const int tid = threadIdx.x;
  const int kmax = min(prm.k_max, st.k);

  // truncated support T_i = top-k_max: mass mu_i and -sum p log p (Eq. 3), not renormalised
  for (int j = tid; j < n_m; j += kT) {
    const float lse = st.lse[j];
    float mu = 0.f, ht = 0.f;
    for (int k = 0; k < kmax; ++k) {
      const float lp = st.topk_logit[size_t(j) * st.k + k] - lse;
      const float p = expf(lp);
      mu += p;
      ht -= p * lp;
    }
    sh_htr[j] = ht;
    sh_feas[j] = prm.mode == RPS_PIVOT_PAPER ? (mu >= prm.tau_pivot) : 0;
    sh_sort[j] = st.H[j];
  }
  if (prm.mode == RPS_PIVOT_BAND) {
    // bitonic sort of H over M (padded with +inf) for the percentile band
    int n2 = 1;
    while (n2 < n_m) n2 <<= 1;
    for (int j = n_m + tid; j < n2; j += kT) sh_sort[j] = INFINITY;
    __syncthreads();
    for (int size = 2; size <= n2; size <<= 1)
      for (int stride = size >> 1; stride > 0; stride >>= 1) {
        for (int x = tid; x < n2 / 2; x += kT) {
          const int lo = 2 * x - (x & (stride - 1));
          const int hi = lo + stride;
          const bool up = (lo & size) == 0;
          const float a = sh_sort[lo], b = sh_sort[hi];
          if ((a > b) == up) { sh_sort[lo] = b; sh_sort[hi] = a; }
        }
        __syncthreads();
      }
    if (tid == 0) {
      for (int e = 0; e < 2; ++e) {
        const float q = (e ? prm.pct_hi : prm.pct_lo) / 100.0f;
        const float idx = q * float(n_m - 1);
        const int lo = min(int(floorf(idx)), n_m - 1);
        const int hi = min(lo + 1, n_m - 1);
        band[e] = sh_sort[lo] + (idx - float(lo)) * (sh_sort[hi] - sh_sort[lo]);
      }
    }
    __syncthreads();
    for (int j = tid; j < n_m; j += kT) {
      const float h = st.H[j];
      sh_feas[j] = h >= band[0] && h <= band[1];
    }
  }
  __syncthreads();

  // the n_pivots feasible rows of largest truncated entropy (lower position first on ties)
  const int n_piv = n_m > 1 ? min(prm.n_pivots, RPS_MAX_PIVOTS) : 0;
  if (tid < RPS_MAX_PIVOTS) chosen[tid] = -1;
  __syncthreads();
  for (int rnd = 0; rnd < n_piv; ++rnd) {
    float bv = -INFINITY;
    int bi = 0x7fffffff;
    for (int j = tid; j < n_m; j += kT)
      if (sh_feas[j] && better(sh_htr[j], m_pos[j], bv, bi)) { bv = sh_htr[j]; bi = m_pos[j]; }
    block_argmax(bv, bi, red_v, red_i);
    for (int j = tid; j < n_m; j += kT)
      if (sh_feas[j] && m_pos[j] == bi && bi != 0x7fffffff) { chosen[rnd] = j; sh_feas[j] = 0; }
    __syncthreads();
  }

  if (tid != 0) return;
  // adaptive candidate sets: v in T_{i*} with p(v) >= r P^max, rank order, capped
  rps_plan& pl = *plan;   // written in place (a private copy would live in scratch memory)
  pl.n_pivots = 0;
  pl.n_branch = 0;
  for (int i = 0; i < RPS_MAX_PIVOTS; ++i) pl.pivot_row[i] = pl.pivot_pos[i] = pl.n_cand[i] = -1;
  for (int i = 0; i < RPS_MAX_BRANCH; ++i) {
    pl.br_pivot[i] = pl.br_row[i] = pl.br_pos[i] = pl.br_token[i] = -1;
    pl.br_logp[i] = 0.f;
  }
  const int cap = min(prm.max_branch, RPS_MAX_BRANCH);
  for (int rnd = 0; rnd < n_piv; ++rnd) {
    const int j = chosen[rnd];
    if (j < 0) break;
    const float lmax = st.lmax[j], lse = st.lse[j];
    int cnt = 0;
    for (int k = 0; k < kmax && cnt < prm.n_cand && pl.n_branch + cnt < cap; ++k) {
      const float lg = st.topk_logit[size_t(j) * st.k + k];
      if (!(expf(lg - lmax) >= prm.r)) break;   // p(v) / P^max is non-increasing in rank
      ++cnt;
    }
    if (cnt < 2) continue;
    const int p = pl.n_pivots++;
    pl.pivot_row[p] = j;
    pl.pivot_pos[p] = m_pos[j];
    pl.n_cand[p] = cnt;
    for (int k = 0; k < cnt; ++k) {
      const int b = pl.n_branch++;
      pl.br_pivot[b] = p;
      pl.br_row[b] = j;
      pl.br_pos[b] = m_pos[j];
      pl.br_token[b] = st.topk_id[size_t(j) * st.k + k];
      pl.br_logp[b] = st.topk_logit[size_t(j) * st.k + k] - lse;
    }
  }
}

__global__ __launch_bounds__(kT) void branch_kernel(const int32_t* __restrict__ tokens, int seq,
                                                    const rps_plan* __restrict__ plan, int anchor_first,
                                                    int32_t* __restrict__ out) {
  const int slot = blockIdx.y;
  const int s = blockIdx.x * kT + threadIdx.x;
  if (s >= seq) return;
  const int b = slot - (anchor_first ? 1 : 0);
  int v = tokens[s];
  if (b >= 0 && b < plan->n_branch && plan->br_pos[b] == s) v = plan->br_token[b];
  out[size_t(slot) * seq + s] = v;
}

// packed lookahead sequence: slot 0 (blockIdx.y) copies the shared sequence,
// slot 1 + b writes branch b's copy of the block at seq + b * B
__global__ __launch_bounds__(kT) void packed_branch_kernel(const int32_t* __restrict__ tokens, int seq,
                                                           const rps_plan* __restrict__ plan, int b0, int B,
                                                           int32_t* __restrict__ out) {
  const int slot = blockIdx.y;
  const int s = blockIdx.x * kT + threadIdx.x;
  if (slot == 0) {
    if (s < seq) out[s] = tokens[s];
    return;
  }
  if (s >= B) return;
  const int b = slot - 1, p = b0 + s;
  int v = tokens[p];
  if (b < plan->n_branch && plan->br_pos[b] == p) v = plan->br_token[b];
  out[seq + size_t(b) * B + s] = v;
}

__global__ __launch_bounds__(kT) void score_kernel(StatsIn anc, StatsIn br, int branch_offset, int n_m,
                                                   const rps_plan* __restrict__ plan,
                                                   const float* __restrict__ anchor_logit, float lambda,
                                                   float* __restrict__ scores, float* __restrict__ deltas,
                                                   rps_decision* __restrict__ dec) {
  __shared__ float sd[RPS_MAX_BRANCH];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nb = n_m > 1 ? plan->n_branch : 0;
  const float inv_n = n_m > 1 ? 1.0f / float(n_m - 1) : 0.f;
  for (int b = wave; b < nb; b += kT / kWave) {
    const int row = plan->br_row[b];
    const float* Hb = br.H + size_t(branch_offset + b) * n_m;
    float dsum = 0.f, hsum = 0.f;
    for (int j = lane; j < n_m; j += kWave) {
      if (j == row) continue;
      const float hb = Hb[j];
      dsum += anc.H[j] - hb;   // entropy reduction relative to the anchor, summed over M minus the pivot
      hsum += hb;
    }
    dsum = wave_sum(dsum);
    hsum = wave_sum(hsum);
    if (lane == 0) {
      const float log_a = anchor_logit ? anchor_logit[b] - anc.lse[row] : plan->br_logp[b];
      const float log_am = anc.lmax[row] - anc.lse[row];   // a_[MASK] = P^max of the anchor
      const float s = -hsum * inv_n + lambda * log_a;
      const float d = dsum * inv_n + lambda * (log_a - log_am);
      sd[b] = d;
      if (scores) scores[b] = s;
      if (deltas) deltas[b] = d;
    }
  }
  __syncthreads();
  if (threadIdx.x != 0) return;
  rps_decision r;
  r.commit = 0;
  r.branch = -1;
  r.pivot_row = r.pivot_pos = r.token = -1;
  r.delta = -INFINITY;
  r.second_delta = -INFINITY;
  r.n_masked = n_m;
  for (int b = 0; b < nb; ++b) {
    if (sd[b] > r.delta) {
      r.second_delta = r.delta;
      r.delta = sd[b];
      r.branch = b;
    } else if (sd[b] > r.second_delta) {
      r.second_delta = sd[b];
    }
  }
  if (r.branch >= 0) {
    r.pivot_row = plan->br_row[r.branch];
    r.pivot_pos = plan->br_pos[r.branch];
    r.token = plan->br_token[r.branch];
    r.commit = r.delta > 0.f;   // a tie with [MASK] abstains
  }
  *dec = r;
}

// Commit the rows flagged in sel (tokens[m_pos[j]] = argmax[j], Eq. 1) after
// the s_nc positions already in committed[], then compact m_pos and the
// statistics (from src into base, possibly in place) to the rows neither
// selected nor equal to `drop`.  Called by all kT threads of the workgroup.
__device__ void commit_compact(int32_t* __restrict__ tokens, int seq, int32_t* __restrict__ m_pos, int n_m,
                               StatsOut base, StatsIn src, const uint8_t* sel, int* pre, int s_drop, int s_nc,
                               int32_t* __restrict__ n_m_out, int32_t* __restrict__ committed,
                               int32_t* __restrict__ n_committed) {
  const int tid = threadIdx.x;
  const int K = base.k;
  // exclusive prefix sums of selected rows (commit order) and of kept rows (new index)
  if (tid == 0) {
    int cs = 0, ks = 0;
    for (int j = 0; j < n_m; ++j) {
      const bool keep = j != s_drop && !sel[j];
      if (sel[j]) {
        committed[s_nc + cs] = m_pos[j];
        tokens[min(max(m_pos[j], 0), seq - 1)] = src.argmax[j];
        ++cs;
      }
      pre[j] = keep ? ks++ : -1;
    }
    *n_m_out = ks;
    *n_committed = s_nc + cs;
  }
  __syncthreads();
  // compaction (possibly in place): each round reads its rows before writing them
  for (int r0 = 0; r0 < n_m; r0 += kT) {
    const int j = r0 + tid;
    const bool act = j < n_m && pre[j] >= 0;
    float h = 0.f, lse = 0.f, lmax = 0.f;
    int am = 0, pos = 0;
    float tl[DLLM_MAX_TOPK];
    int tid_[DLLM_MAX_TOPK];
    if (act) {
      h = src.H[j];
      lse = src.lse[j];
      lmax = src.lmax[j];
      am = src.argmax[j];
      pos = m_pos[j];
#pragma unroll
      for (int k = 0; k < DLLM_MAX_TOPK; ++k)
        if (k < K) {
          tl[k] = src.topk_logit[size_t(j) * src.k + k];
          tid_[k] = src.topk_id[size_t(j) * src.k + k];
        }
    }
    __syncthreads();
    if (act) {
      const int nj = pre[j];
      base.H[nj] = h;
      base.lse[nj] = lse;
      base.lmax[nj] = lmax;
      base.argmax[nj] = am;
      m_pos[nj] = pos;
#pragma unroll
      for (int k = 0; k < DLLM_MAX_TOPK; ++k)
        if (k < K) {
          base.topk_logit[size_t(nj) * K + k] = tl[k];
          base.topk_id[size_t(nj) * K + k] = tid_[k];
        }
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(kT) void commit_kernel(int32_t* __restrict__ tokens, int seq, int32_t* __restrict__ m_pos,
                                                    int n_m,
                                                    StatsOut base, const rps_decision* __restrict__ dec,
                                                    StatsIn brs, int branch_offset, StatsIn anc, int has_anchor,
                                                    float tau, int32_t* __restrict__ n_m_out,
                                                    int32_t* __restrict__ committed,
                                                    int32_t* __restrict__ n_committed) {
  __shared__ uint8_t sel[kMaxM];
  __shared__ int pre[kMaxM];
  __shared__ int wsum[kT / kWave];
  __shared__ float red_v[4];
  __shared__ int red_i[4];
  __shared__ int s_drop, s_nc;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  // source of the carried statistics
  StatsIn src{base.H, base.lse, base.lmax, base.argmax, base.topk_id, base.topk_logit, base.k};
  int drop = -1;
  if (dec) {
    if (dec->commit) {
      const size_t off = size_t(branch_offset + dec->branch) * n_m;
      src = StatsIn{brs.H + off, brs.lse + off, brs.lmax + off, brs.argmax + off,
                    brs.topk_id + off * brs.k, brs.topk_logit + off * brs.k, brs.k};
      drop = dec->pivot_row;
    } else if (has_anchor) {
      src = anc;
    }
  }
  if (tid == 0) {
    s_nc = 0;
    s_drop = drop;
    if (drop >= 0) {
      tokens[min(max(dec->pivot_pos, 0), seq - 1)] = dec->token;
      committed[0] = dec->pivot_pos;
      s_nc = 1;
    }
  }
  // confidence-aware commit on the carried statistics
  int n_sel = 0;
  for (int j = tid; j < n_m; j += kT) {
    bool s = false;
    if (tau >= 0.f && j != drop) s = expf(src.lmax[j] - src.lse[j]) >= tau;
    sel[j] = s;
  }
  __syncthreads();
  if (tau >= 0.f) {
    int c = 0;
    for (int j = tid; j < n_m; j += kT) c += sel[j];
    for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o, 64);
    if (lane == 0) wsum[wave] = c;
    __syncthreads();
    n_sel = wsum[0] + wsum[1] + wsum[2] + wsum[3];
    __syncthreads();
    if (n_sel == 0 && n_m - (drop >= 0 ? 1 : 0) > 0) {  // fallback: the single most confident row
      float bv = -INFINITY;
      int bi = 0x7fffffff;
      for (int j = tid; j < n_m; j += kT)
        if (j != drop) {
          const float pm = expf(src.lmax[j] - src.lse[j]);
          if (better(pm, j, bv, bi)) { bv = pm; bi = j; }
        }
      block_argmax(bv, bi, red_v, red_i);
      if (tid == 0) sel[bi] = 1;
      n_sel = 1;
      __syncthreads();
    }
  }
  commit_compact(tokens, seq, m_pos, n_m, base, src, sel, pre, s_drop, s_nc, n_m_out, committed, n_committed);
}

// Baseline schedulers of Eq. 2 (first two cases): commit the k rows of
// highest confidence (key log P^max = lmax - lse) or of lowest entropy
// (key -H); ties go to the lower row, i.e. the lower position.  A row is
// selected iff fewer than k rows beat it, counted against every row in LDS.
__global__ __launch_bounds__(kT) void sched_kernel(int32_t* __restrict__ tokens, int seq, int32_t* __restrict__ m_pos,
                                                   int n_m, StatsOut base, int rule, int k,
                                                   int32_t* __restrict__ n_m_out, int32_t* __restrict__ committed,
                                                   int32_t* __restrict__ n_committed) {
  __shared__ float key[kMaxM];
  __shared__ uint8_t sel[kMaxM];
  __shared__ int pre[kMaxM];
  const int tid = threadIdx.x;
  for (int j = tid; j < n_m; j += kT) key[j] = rule == SCHED_LOW_ENTROPY ? -base.H[j] : base.lmax[j] - base.lse[j];
  __syncthreads();
  for (int j = tid; j < n_m; j += kT) {
    const float v = key[j];
    int rank = 0;
    for (int o = 0; o < n_m; ++o) rank += better(key[o], o, v, j);
    sel[j] = rank < k;
  }
  __syncthreads();
  const StatsIn src{base.H, base.lse, base.lmax, base.argmax, base.topk_id, base.topk_logit, base.k};
  commit_compact(tokens, seq, m_pos, n_m, base, src, sel, pre, -1, 0, n_m_out, committed, n_committed);
}

StatsIn to_in(const StatsOut& s) { return StatsIn{s.H, s.lse, s.lmax, s.argmax, s.topk_id, s.topk_logit, s.k}; }

}  // namespace

hipError_t rps_select(const StatsOut& base, const int32_t* m_pos, int n_m, const rps_params& prm, rps_plan* plan,
                      hipStream_t s) {
  hipLaunchKernelGGL(select_kernel, dim3(1), dim3(kT), 0, s, to_in(base), m_pos, n_m, prm, plan);
  return hipGetLastError();
}

hipError_t rps_branches(const int32_t* tokens, int seq, const rps_plan* plan, int anchor_first, int capacity,
                        int32_t* out, hipStream_t s) {
  hipLaunchKernelGGL(branch_kernel, dim3(cdiv(seq, kT), capacity), dim3(kT), 0, s, tokens, seq, plan, anchor_first,
                     out);
  return hipGetLastError();
}

hipError_t rps_branches_packed(const int32_t* tokens, int seq, const rps_plan* plan, int b0, int B, int capacity,
                               int32_t* out, hipStream_t s) {
  hipLaunchKernelGGL(packed_branch_kernel, dim3(cdiv(std::max(seq, B), kT), 1 + capacity), dim3(kT), 0, s, tokens,
                     seq, plan, b0, B, out);
  return hipGetLastError();
}

hipError_t rps_score(const StatsOut& anchor, const StatsOut& branches, int branch_offset, int n_m,
                     const rps_plan* plan, const float* anchor_logit, float lambda, float* scores, float* deltas,
                     rps_decision* dec, hipStream_t s) {
  hipLaunchKernelGGL(score_kernel, dim3(1), dim3(kT), 0, s, to_in(anchor), to_in(branches), branch_offset, n_m, plan,
                     anchor_logit, lambda, scores, deltas, dec);
  return hipGetLastError();
}

hipError_t rps_commit_step(int32_t* tokens, int seq, int32_t* m_pos, int n_m, const StatsOut& base, const rps_decision* dec,
                           const StatsOut* branches, int branch_offset, const StatsOut* anchor, float tau,
                           int32_t* n_m_out, int32_t* committed, int32_t* n_committed, hipStream_t s) {
  const StatsIn br = branches ? to_in(*branches) : StatsIn{};
  const StatsIn an = anchor ? to_in(*anchor) : StatsIn{};
  hipLaunchKernelGGL(commit_kernel, dim3(1), dim3(kT), 0, s, tokens, seq, m_pos, n_m, base, dec, br, branch_offset, an,
                     anchor ? 1 : 0, tau, n_m_out, committed, n_committed);
  return hipGetLastError();
}

hipError_t sched_commit_step(int32_t* tokens, int seq, int32_t* m_pos, int n_m, const StatsOut& st, int rule, int k,
                            int32_t* n_m_out, int32_t* committed, int32_t* n_committed, hipStream_t s) {
  hipLaunchKernelGGL(sched_kernel, dim3(1), dim3(kT), 0, s, tokens, seq, m_pos, n_m, st, rule, k, n_m_out, committed,
                     n_committed);
  return hipGetLastError();
}

}  // namespace dllm
