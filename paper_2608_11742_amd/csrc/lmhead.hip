// LM head fused with the per-position vocabulary statistics the scheduler
// needs (entropy, log-sum-exp, max logit, argmax, top-K).  The [R][V] logits
// never leave the chip.
//
// Pass 1 (lmhead_kernel): a workgroup owns 128 hidden rows and one slice of
// the vocabulary.  For each 256-token vocabulary tile it runs the MFMA
// mainloop, scales the logits, stages the 128x256 fp32 tile in LDS and lets
// 4 threads per row scan 64 logits each, updating a running max m,
// s = sum exp(l - m), t = sum exp(l - m) (l - m) (m and t in log2 units
// while scanning, natural units in the partials) and a sorted top-16.  At
// the end of its slice every thread writes its partial state.
// Pass 2 (merge_kernel): one workgroup per row merges all partials:
//   M = max m_p, S = sum s_p e^(m_p - M), T = sum e^(m_p - M) (t_p + (m_p - M) s_p)
//   lse = M + log S, H = log S - T / S, lmax = M,
// and a 64-way merge of the sorted partial top-16 lists.
#include <algorithm>
#include <type_traits>

#include "kernels.h"
#include "mainloop.h"

namespace dllm {

namespace {

constexpr int kCols = 256;                               // vocabulary tile
constexpr int kThreads = 512;
constexpr int kK = DLLM_TOPK_REG;
constexpr int kSegCols = 64;                             // logits per scan thread per pass
constexpr int kSegStride = kSegCols * 4 + 16;            // padded segment bytes
// Workgroups of a launch: one per CU (the 256-row tile's LDS holds one), each
// walking its vocabulary slice.  Two rounds of half-length slices measured
// 4-6% slower at 512 and 4096 rows: every slice pays its first tile, where
// the empty top-16 lists make many logits candidates, and the merge folds
// twice the partials.
constexpr int kTargetWg = 256;
constexpr float kLog2e = 1.4426950408889634f, kLn2 = 0.6931471805599453f;

// BM rows per workgroup: 256 (8 waves of 64 x 128, the projection GEMMs'
// tile) when there are more than 128 rows, else 128 (8 waves of 64 x 64).
// kSegs scan threads per row, each scanning 64 logits per pass; a pass
// stages kSegs * 64 columns of the fp32 logit tile in LDS.
// The MFMA blocks are computed transposed (TRANS), so that a lane holds 4
// consecutive logits of one row and stages them with one 16-byte LDS write;
// bf16 256-row tiles take the two-group mainloop of the projections;
// 128-row tiles (few rows: the vocabulary streams from HBM) the early-release
// TileMma schedule.
template <typename T, int BM>
struct LmCfg {
  using TM = std::conditional_t<BM == 256 && std::is_same_v<T, bf16_t>, PingPongMma<T, true>,
                                TileMma<T, BM, kCols, BM == 256 ? 4 : 2, BM == 256 ? 2 : 4, true, BM == 128>>;
  static constexpr int kSegs = kThreads / BM;
  static constexpr int kPassCols = kSegs * kSegCols;
  static constexpr int kPasses = kCols / kPassCols;
  static constexpr int kRowStride = kSegs * kSegStride + 16;   // padded row bytes
  static constexpr int kStageBytes = BM * kRowStride;
  static constexpr int kSmem = TM::kSmem > kStageBytes ? TM::kSmem : kStageBytes;
  static constexpr int kBoundRank = kK / kSegs - 1;            // see the pruning bound below
  static_assert(kPasses == 1 || kPassCols == TM::kWTN, "a pass is the whole tile or one wave column");
};

int tile_rows(int R) { return R > 128 ? 256 : 128; }

struct Partials {
  float* m;
  float* s;
  float* t;
  float* tv;     // [R][P][16]
  int32_t* ti;   // [R][P][16]
  int P;
};

__device__ __forceinline__ void topk_insert(float (&tv)[kK], int (&ti)[kK], float v, int id) {
  float cv = v;
  int ci = id;
#pragma unroll
  for (int k = 0; k < kK; ++k) {
    const bool gt = better(cv, ci, tv[k], ti[k]);
    const float ov = tv[k];
    const int oi = ti[k];
    tv[k] = gt ? cv : ov;
    ti[k] = gt ? ci : oi;
    cv = gt ? ov : cv;
    ci = gt ? oi : ci;
  }
}

template <typename T, int BM>
__global__ __launch_bounds__(kThreads, 1) void lmhead_kernel(const T* __restrict__ Hs, const T* __restrict__ W, int R,
                                                             int d, int V, const float* __restrict__ row_scale,
                                                             const int32_t* __restrict__ rs_idx, int rs_n, int rs_lim,
                                                             float scale, int mask_id, int row_tiles,
                                                             int n_slices,
                                                             int vtiles, Partials part) {
  using Cfg = LmCfg<T, BM>;
  using TM = typename Cfg::TM;
  constexpr int kSegs = Cfg::kSegs, kRowStride = Cfg::kRowStride;
  __shared__ __attribute__((aligned(16))) uint8_t smem[Cfg::kSmem];

  // XCD-contiguous ids, walked in groups of 8 row tiles: the 32 workgroups an
  // XCD runs at a time cover 8 row tiles x 4 vocabulary slices, so each step
  // of their vocabulary loops fetches 12 operand panels into that XCD's L2
  // (16 row tiles x 2 slices would fetch 18)
  int rt, slice;
  map_tile(blockIdx.x, gridDim.x, row_tiles, n_slices, 8, rt, slice);
  const int t_begin = int((long long)slice * vtiles / n_slices);
  const int t_end = int((long long)(slice + 1) * vtiles / n_slices);
  const int m0 = rt * BM;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  constexpr int kWavesN = kCols / TM::kWTN;
  const int wm = wave / kWavesN, wn = wave % kWavesN;
  // scan role: row tid / kSegs, segment tid % kSegs
  const int srow = tid / kSegs, sseg = tid % kSegs;
  float m = -INFINITY, s = 0.f, t = 0.f;
  // This thread's sorted top 16.  With 256-row tiles the mainloop needs
  // nearly every register, so between tiles the list lives in the thread's
  // partials slot of the workspace (loaded before the scan, stored after it);
  // with 128-row tiles it stays in registers.
  constexpr bool kListInMemory = BM == 256;
  const int row = m0 + srow;
  const bool own_row = row < R;   // rows past R scan clamped copies and are discarded
  size_t slot = size_t(min(row, R - 1)) * part.P + size_t(slice) * kSegs + sseg;
  float tv[kK];
  int ti[kK];
#pragma unroll
  for (int k = 0; k < kK; ++k) { tv[k] = -INFINITY; ti[k] = 0x7fffffff; }
  // Pruning bound of the row, shared by its kSegs scan threads: the worst
  // (by value, then id) of their (16 / kSegs)-th best entries.  Each thread
  // holds 16 / kSegs entries at least as good as that, so at least 16
  // entries of the row are at least as good as the bound, and a logit that
  // is not strictly better cannot reach the row's top 16.  It rises about as
  // fast as the row's 16th best over all its segments, kSegs times faster
  // than a thread's own 16th best, which keeps the (wave-divergent)
  // insertions rare.
  float bv = -INFINITY;
  int bi = 0x7fffffff;

  // logit scale of this thread's scan row
  const int srow_c = min(row, R - 1);
  auto row_logit_scale = [&]() {
    return scale *
           (row_scale ? row_scale[rs_idx ? min(max(rs_idx[srow_c % rs_n], 0), rs_lim - 1) : srow_c % rs_n] : 1.0f);
  };
  float rs_row = row_logit_scale();

  // the bound from the kSegs threads of this row (consecutive lanes)
  auto refresh_bound = [&]() {
    float v = tv[Cfg::kBoundRank];
    int i = ti[Cfg::kBoundRank];
#pragma unroll
    for (int x = 1; x < kSegs; x <<= 1) {
      const float ov = __shfl_xor(v, x, 64);
      const int oi = __shfl_xor(i, x, 64);
      if (better(v, i, ov, oi)) { v = ov; i = oi; }
    }
    bv = v;
    bi = i;
  };

  const uint32_t row_bytes = uint32_t(d) * sizeof(T);
  for (int vt = t_begin; vt < t_end; ++vt) {
    // opaque per tile: keeps the compiler from hoisting the slot addresses
    // out of the tile loop, where they would stay live across the mainloop
    if constexpr (kListInMemory) asm volatile("" : "+v"(slot));
    const int n0 = vt * kCols;
    auto a_off = [&](int r) -> uint32_t { return uint32_t(min(m0 + r, R - 1)) * row_bytes; };
    auto b_off = [&](int r) -> uint32_t { return uint32_t(min(n0 + r, V - 1)) * row_bytes; };
    f32x4 acc[TM::kFM][TM::kFN];
    TM::run(smem, reinterpret_cast<const uint8_t*>(Hs), reinterpret_cast<const uint8_t*>(W), a_off, b_off,
            d / TM::kKPerStage, acc);
    if constexpr (kListInMemory) {
      if (vt > t_begin && own_row) {
        m = part.m[slot] * kLog2e;   // log2 units while scanning
        s = part.s[slot];
        t = part.t[slot] * kLog2e;
#pragma unroll
        for (int k = 0; k < kK; ++k) {
          tv[k] = part.tv[slot * kK + k];
          ti[k] = part.ti[slot * kK + k];
        }
      } else {
        m = -INFINITY;
        s = t = 0.f;
#pragma unroll
        for (int k = 0; k < kK; ++k) { tv[k] = -INFINITY; ti[k] = 0x7fffffff; }
      }
      refresh_bound();
      rs_row = row_logit_scale();
    }
#pragma unroll
    for (int pass = 0; pass < Cfg::kPasses; ++pass) {
    // stage this pass's scaled logits: LDS row r, pass column c at
    // r * kRowStride + (c / 64) * kSegStride + (c % 64) * 4
    if (Cfg::kPasses == 1 || wn == pass) {
#pragma unroll
      for (int mi = 0; mi < TM::kFM; ++mi)
#pragma unroll
        for (int ni = 0; ni < TM::kFN; ++ni) {
          // (transposed blocks) row 16 mi + lane % 16, columns 16 ni + 4 (lane / 16) + 0..3
          const int r = wm * TM::kWTM + mi * 16 + (lane & 15);
          const int c = wn * TM::kWTN + ni * 16 + 4 * (lane >> 4) - pass * Cfg::kPassCols;
          *reinterpret_cast<f32x4*>(smem + r * kRowStride + (c >> 6) * kSegStride + (c & 63) * 4) = acc[mi][ni];
        }
    }
    __syncthreads();
    // scan 64 logits of row srow: running statistics, and a bit mask of the
    // logits that may beat the pruning bound (candidates for the top 16)
    const uint8_t* base = smem + srow * kRowStride + sseg * kSegStride;
    const int c0 = n0 + pass * Cfg::kPassCols + sseg * kSegCols;
    const bool all_ok = c0 + kSegCols <= V && (mask_id < c0 || mask_id >= c0 + kSegCols);
    if (vt == t_begin && pass == 0) {
      // The slice's top-16 lists are still empty, which would make every
      // logit a candidate.  Seed the bound instead: each thread takes the
      // smallest of the maxima of its 8 groups of 8 logits (8 logits are at
      // least that large), the row the smallest over its kSegs threads, so at
      // least 16 logits of the row are at least as large as the bound and no
      // smaller logit can reach the row's top 16.
      float seed = INFINITY;
#pragma unroll
      for (int g8 = 0; g8 < kSegCols; g8 += 8) {
        float gm = -INFINITY;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int col = c0 + g8 + e;
          const float v = *reinterpret_cast<const float*>(base + (g8 + e) * 4) * rs_row;
          if (all_ok || (col < V && col != mask_id)) gm = fmaxf(gm, v);
        }
        seed = fminf(seed, gm);
      }
#pragma unroll
      for (int x = 1; x < kSegs; x <<= 1) seed = fminf(seed, __shfl_xor(seed, x, 64));
      if (better(seed, 0x7fffffff, bv, bi)) {   // only ever raises the bound
        bv = seed;
        bi = 0x7fffffff;
      }
    }
    uint64_t cand = 0;
    if (__all(all_ok)) {
      // Every logit of the wave's segments is valid: branch-free scan in
      // log2 units (x = logit * log2 e): one FMA, one exp2 and one FMA per
      // logit; the reference max moves by selects.  Candidates are the
      // logits with x at least the bound in log2 units less a relative
      // 1e-6 (x and the bound round differently, by a few ulp at most), a
      // superset of those that beat the bound; the insertion below checks
      // each one exactly.
      const float c2 = rs_row * kLog2e;
      const float b2 = bv * kLog2e;
      const float bv2 = own_row ? b2 - fabsf(b2) * 1e-6f : INFINITY;
#pragma unroll
      for (int c4 = 0; c4 < kSegCols; c4 += 4) {
        const float4 v4 = *reinterpret_cast<const float4*>(base + c4 * 4);
        const float x[4] = {v4.x * c2, v4.y * c2, v4.z * c2, v4.w * c2};
        const float gmax = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
        const float mnew = fmaxf(m, gmax);
        const float alpha = __builtin_amdgcn_exp2f(m - mnew);   // 1 if unchanged, 0 from -inf
        const float d = alpha == 0.f ? 0.f : m - mnew;
        t = alpha * (t + d * s);
        s = alpha * s;
        m = mnew;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float y = x[e] - m;
          const float ex = __builtin_amdgcn_exp2f(y);
          s += ex;
          t = fmaf(ex, y, t);
          cand |= uint64_t(x[e] >= bv2) << (c4 + e);
        }
      }
    } else {
#pragma unroll
    for (int c4 = 0; c4 < kSegCols; c4 += 4) {
      const float4 v4 = *reinterpret_cast<const float4*>(base + c4 * 4);
      const float vv[4] = {v4.x * rs_row, v4.y * rs_row, v4.z * rs_row, v4.w * rs_row};
      bool ok[4];
      float cmax = -INFINITY;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int col = c0 + c4 + e;
        ok[e] = all_ok || (col < V && col != mask_id);
        if (ok[e]) cmax = fmaxf(cmax, vv[e] * kLog2e);
      }
      if (cmax > m) {  // rescale the running sums to the new max (log2 units)
        if (m > -INFINITY) {
          const float alpha = __builtin_amdgcn_exp2f(m - cmax);
          t = alpha * (t + (m - cmax) * s);
          s = alpha * s;
        }
        m = cmax;
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (!ok[e]) continue;
        const float x = vv[e] * kLog2e - m;
        const float ex = __builtin_amdgcn_exp2f(x);
        s += ex;
        t += ex * x;
        if (own_row && better(vv[e], c0 + c4 + e, bv, bi)) cand |= uint64_t(1) << (c4 + e);
      }
    }
    }
    // insert the candidates; the wave loops as often as its busiest lane has candidates
    while (__any(cand != 0)) {
      if (cand) {
        const int pos = __builtin_ctzll(cand);
        cand &= cand - 1;
        const float v = *reinterpret_cast<const float*>(base + pos * 4) * rs_row;
        if (better(v, c0 + pos, tv[kK - 1], ti[kK - 1])) topk_insert(tv, ti, v, c0 + pos);
      }
    }
    // the next pass prunes with the bound these insertions raised
    if (pass + 1 < Cfg::kPasses) refresh_bound();
    __syncthreads();
    }
    if constexpr (!kListInMemory) refresh_bound();
    if (kListInMemory && own_row) {
      part.m[slot] = m * kLn2;   // natural units in the partials
      part.s[slot] = s;
      part.t[slot] = t * kLn2;
#pragma unroll
      for (int k = 0; k < kK; ++k) {
        part.tv[slot * kK + k] = tv[k];
        part.ti[slot * kK + k] = ti[k];
      }
    }
  }
  if (own_row && !kListInMemory) {
    part.m[slot] = m * kLn2;
    part.s[slot] = s;
    part.t[slot] = t * kLn2;
    {
#pragma unroll
      for (int k = 0; k < kK; ++k) {
        part.tv[slot * kK + k] = tv[k];
        part.ti[slot * kK + k] = ti[k];
      }
    }
  }
}

// One workgroup of W = blockDim.x / 64 waves per row (W grows with the number
// of partials, so that rows with many vocabulary slices merge in parallel).
// Every lane folds a strided share of the row's partials into (S, T) and a
// sorted top-16; each wave merges its lanes' lists into its own top-16 by
// repeated wave-wide argmax; the waves' lists and sums meet in LDS and wave 0
// merges them the same way.
__global__ __launch_bounds__(512) void merge_kernel(Partials part, int R, StatsOut out) {
  constexpr int kMaxW = 8;
  __shared__ float red_m[kMaxW], red_s[kMaxW], red_t[kMaxW];
  __shared__ float lv[kMaxW][kK];
  __shared__ int li[kMaxW][kK];
  const int row = blockIdx.x;
  const int W = blockDim.x >> 6, wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (row >= R) return;
  const size_t base = size_t(row) * part.P;
  float M = -INFINITY;
  for (int p = threadIdx.x; p < part.P; p += blockDim.x) M = fmaxf(M, part.m[base + p]);
  M = wave_max(M);
  if (lane == 0) red_m[wave] = M;
  __syncthreads();
  M = red_m[0];
  for (int w = 1; w < W; ++w) M = fmaxf(M, red_m[w]);
  float S = 0.f, Tt = 0.f;
  float tv[kK];
  int ti[kK];
#pragma unroll
  for (int k = 0; k < kK; ++k) { tv[k] = -INFINITY; ti[k] = 0x7fffffff; }
  for (int p = threadIdx.x; p < part.P; p += blockDim.x) {
    const float mp = part.m[base + p];
    if (mp == -INFINITY) continue;  // a partial that saw no valid logit
    const float w = fast_exp(mp - M);
    const float sp = part.s[base + p];
    S += w * sp;
    Tt += w * (part.t[base + p] + (mp - M) * sp);
    const float* pv = part.tv + (base + p) * kK;
    const int32_t* pi = part.ti + (base + p) * kK;
#pragma unroll
    for (int k = 0; k < kK; ++k) {
      const float v = pv[k];
      const int i = pi[k];
      if (better(v, i, tv[kK - 1], ti[kK - 1])) topk_insert(tv, ti, v, i);
    }
  }
  S = wave_sum(S);
  Tt = wave_sum(Tt);
  // 64-way merge of the lanes' sorted lists: the wave-wide best head is taken n times
  auto merge_lanes = [&](int n, auto&& emit) {
    for (int k = 0; k < n; ++k) {
      float v = tv[0];
      int i = ti[0];
      wave_argmax(v, i);
      emit(k, v, i);
      if (ti[0] == i) {  // ids are unique: exactly one lane owns the winner; pop it
#pragma unroll
        for (int j = 0; j < kK - 1; ++j) { tv[j] = tv[j + 1]; ti[j] = ti[j + 1]; }
        tv[kK - 1] = -INFINITY;
        ti[kK - 1] = 0x7fffffff;
      }
    }
  };
  if (W > 1) {
    merge_lanes(kK, [&](int k, float v, int i) {
      if (lane == 0) { lv[wave][k] = v; li[wave][k] = i; }
    });
    if (lane == 0) { red_s[wave] = S; red_t[wave] = Tt; }
    __syncthreads();
    if (wave != 0) return;
    S = red_s[0];
    Tt = red_t[0];
    for (int w = 1; w < W; ++w) { S += red_s[w]; Tt += red_t[w]; }
#pragma unroll
    for (int k = 0; k < kK; ++k) {
      tv[k] = lane < W ? lv[lane][k] : -INFINITY;
      ti[k] = lane < W ? li[lane][k] : 0x7fffffff;
    }
  }
  merge_lanes(out.k, [&](int k, float v, int i) {
    if (lane == 0) {
      out.topk_id[size_t(row) * out.k + k] = i;
      out.topk_logit[size_t(row) * out.k + k] = v;
      if (k == 0) out.argmax[row] = i;
    }
  });
  if (lane == 0) {
    const float logS = logf(S);
    out.lmax[row] = M;
    out.lse[row] = M + logS;
    out.H[row] = logS - Tt / S;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void probe_kernel(const T* __restrict__ Hs, const T* __restrict__ W, int d, int V,
                                                    int R, const int32_t* __restrict__ row,
                                                    const int32_t* __restrict__ tok, int n,
                                                    const float* __restrict__ row_scale,
                                                    const int32_t* __restrict__ rs_idx, int n_pos, int rs_lim,
                                                    float scale, float* __restrict__ out) {
  const int p = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (p >= n) return;
  const int r = min(max(row[p], 0), R - 1);
  const T* h = Hs + size_t(r) * d;
  const T* w = W + size_t(min(max(tok[p], 0), V - 1)) * d;
  float acc = 0.f;
  for (int c = lane; c < d; c += 64) acc += load_f(h + c) * load_f(w + c);
  acc = wave_sum(acc);
  if (lane == 0) out[p] = acc * scale * (row_scale ? row_scale[rs_idx ? min(max(rs_idx[r % n_pos], 0), rs_lim - 1) : r % n_pos] : 1.0f);
}

int slices_for(int R, int V) {
  const int rt = cdiv(R, tile_rows(R)), vt = cdiv(V, kCols);
  return std::max(1, std::min(vt, cdiv(kTargetWg, rt)));
}

int partials_per_row(int R, int V) { return slices_for(R, V) * (kThreads / tile_rows(R)); }

Partials carve(void* ws, int R, int P) {
  Partials pt;
  uint8_t* p = static_cast<uint8_t*>(ws);
  const size_t n = size_t(R) * P;
  pt.m = reinterpret_cast<float*>(p);
  pt.s = pt.m + n;
  pt.t = pt.s + n;
  pt.tv = pt.t + n;
  pt.ti = reinterpret_cast<int32_t*>(pt.tv + n * kK);
  pt.P = P;
  return pt;
}

}  // namespace

size_t lmhead_workspace(int R, int V) {
  const size_t P = size_t(partials_per_row(R, V));
  return size_t(R) * P * (3 + 2 * kK) * 4 + 256;
}

hipError_t lmhead_partials(int dtype, const void* h, const void* w, int R, int d, int V, const float* row_scale,
                           const int32_t* rs_idx, int rs_n, int rs_lim, float scale, int mask_id, void* ws,
                           hipStream_t s) {
  if (d <= 0 || d % (dtype ? 64 : 32)) return hipErrorInvalidValue;   // the mainloop runs stages in pairs
  const int ns = slices_for(R, V);
  const int bm = tile_rows(R);
  const int rt = cdiv(R, bm), vt = cdiv(V, kCols);
  Partials part = carve(ws, R, partials_per_row(R, V));
  const int grid = rt * ns;
  auto go = [&](auto kern, auto* hp, auto* wp) {
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kThreads), 0, s, hp, wp, R, d, V, row_scale, rs_idx, rs_n, rs_lim,
                       scale, mask_id, rt, ns, vt, part);
  };
  const bf16_t* hb = static_cast<const bf16_t*>(h);
  const bf16_t* wb = static_cast<const bf16_t*>(w);
  const float* hf = static_cast<const float*>(h);
  const float* wf = static_cast<const float*>(w);
  if (dtype)
    bm == 256 ? go(lmhead_kernel<bf16_t, 256>, hb, wb) : go(lmhead_kernel<bf16_t, 128>, hb, wb);
  else
    bm == 256 ? go(lmhead_kernel<float, 256>, hf, wf) : go(lmhead_kernel<float, 128>, hf, wf);
  return hipGetLastError();
}

hipError_t lmhead_merge(int R, int V, const StatsOut& out, void* ws, hipStream_t s) {
  Partials part = carve(ws, R, partials_per_row(R, V));
  const int waves = std::min(8, std::max(1, cdiv(part.P, 128)));
  hipLaunchKernelGGL(merge_kernel, dim3(R), dim3(64 * waves), 0, s, part, R, out);
  return hipGetLastError();
}

hipError_t probe_logits(int dtype, const void* h, const void* w, int d, int V, int R, const int32_t* row,
                        const int32_t* tok, int n, const float* row_scale, const int32_t* rs_idx, int n_pos,
                        int rs_lim, float scale, float* out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (dtype)
    hipLaunchKernelGGL(probe_kernel<bf16_t>, dim3(cdiv(n, 4)), dim3(256), 0, s, static_cast<const bf16_t*>(h),
                       static_cast<const bf16_t*>(w), d, V, R, row, tok, n, row_scale, rs_idx, n_pos, rs_lim, scale, out);
  else
    hipLaunchKernelGGL(probe_kernel<float>, dim3(cdiv(n, 4)), dim3(256), 0, s, static_cast<const float*>(h),
                       static_cast<const float*>(w), d, V, R, row, tok, n, row_scale, rs_idx, n_pos, rs_lim, scale, out);
  return hipGetLastError();
}

}  // namespace dllm
