// LM head fused with the per-position vocabulary statistics the scheduler
// needs (entropy, log-sum-exp, max logit, argmax, top-K).  The [R][V] logits
// never leave the chip.
//
// Pass 1 (lmhead_kernel): a workgroup owns 128 hidden rows and one slice of
// the vocabulary.  For each 256-token vocabulary tile it runs the MFMA
// mainloop, scales the logits, stages the 128x256 fp32 tile in LDS and lets
// 4 threads per row scan 64 logits each, updating a running max m,
// s = sum exp(l - m), t = sum exp(l - m) (l - m) and a sorted top-16 held in
// registers.  At the end of its slice every thread writes its partial state.
// Pass 2 (merge_kernel): one wave per row merges all partials:
//   M = max m_p, S = sum s_p e^(m_p - M), T = sum e^(m_p - M) (t_p + (m_p - M) s_p)
//   lse = M + log S, H = log S - T / S, lmax = M,
// and a 64-way merge of the sorted partial top-16 lists.
#include <algorithm>

#include "kernels.h"
#include "mainloop.h"

namespace dllm {

namespace {

constexpr int kRows = 128, kCols = 256;
constexpr int kThreads = 512;
constexpr int kK = DLLM_TOPK_REG;
constexpr int kSegs = 4;                                 // threads per row
constexpr int kSegCols = kCols / kSegs;                  // 64 logits per thread per tile
constexpr int kSegStride = kSegCols * 4 + 16;            // padded segment bytes
constexpr int kRowStride = kSegs * kSegStride + 16;      // padded row bytes
constexpr int kStageBytes = kRows * kRowStride;
constexpr int kTargetWg = 512;

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

template <typename T>
__global__ __launch_bounds__(kThreads, 2) void lmhead_kernel(const T* __restrict__ Hs, const T* __restrict__ W, int R,
                                                             int d, int V, const float* __restrict__ row_scale,
                                                             const int32_t* __restrict__ rs_idx, int rs_n, int rs_lim,
                                                             float scale, int mask_id, int row_tiles,
                                                             int n_slices,
                                                             int vtiles, Partials part) {
  using TM = TileMma<T, kRows, kCols, 2, 4>;
  constexpr int kSmem = TM::kSmem > kStageBytes ? TM::kSmem : kStageBytes;
  __shared__ __attribute__((aligned(16))) uint8_t smem[kSmem];

  // XCD-contiguous ids; all row tiles of one vocabulary slice run on one XCD
  const int nwg = gridDim.x, id = blockIdx.x;
  const int q = nwg / 8, rr = nwg % 8, xcd = id % 8, local = id / 8;
  const int lin = xcd < rr ? xcd * (q + 1) + local : rr * (q + 1) + (xcd - rr) * q + local;
  const int slice = lin / row_tiles, rt = lin % row_tiles;
  const int t_begin = int((long long)slice * vtiles / n_slices);
  const int t_end = int((long long)(slice + 1) * vtiles / n_slices);
  const int m0 = rt * kRows;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / 4, wn = wave % 4;
  // scan role: row tid / 4, segment tid % 4
  const int srow = tid >> 2, sseg = tid & 3;
  float m = -INFINITY, s = 0.f, t = 0.f;
  float tv[kK];
  int ti[kK];
#pragma unroll
  for (int k = 0; k < kK; ++k) { tv[k] = -INFINITY; ti[k] = 0x7fffffff; }

  // per-row logit scale of the rows this lane writes in the MFMA layout
  float rs[TM::kFM][4];
#pragma unroll
  for (int mi = 0; mi < TM::kFM; ++mi)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = min(m0 + wm * TM::kWTM + mi * 16 + 4 * (lane >> 4) + i, R - 1);
      rs[mi][i] = scale * (row_scale ? row_scale[rs_idx ? min(max(rs_idx[row % rs_n], 0), rs_lim - 1) : row % rs_n] : 1.0f);
    }

  const uint32_t row_bytes = uint32_t(d) * sizeof(T);
  for (int vt = t_begin; vt < t_end; ++vt) {
    const int n0 = vt * kCols;
    auto a_off = [&](int r) -> uint32_t { return uint32_t(min(m0 + r, R - 1)) * row_bytes; };
    auto b_off = [&](int r) -> uint32_t { return uint32_t(min(n0 + r, V - 1)) * row_bytes; };
    f32x4 acc[TM::kFM][TM::kFN];
    TM::run(smem, reinterpret_cast<const uint8_t*>(Hs), reinterpret_cast<const uint8_t*>(W), a_off, b_off,
            d / TM::kKPerStage, acc);
    // stage scaled logits: LDS row r, column c at r * kRowStride + (c / 64) * kSegStride + (c % 64) * 4
#pragma unroll
    for (int mi = 0; mi < TM::kFM; ++mi)
#pragma unroll
      for (int ni = 0; ni < TM::kFN; ++ni)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = wm * TM::kWTM + mi * 16 + 4 * (lane >> 4) + i;
          const int c = wn * TM::kWTN + ni * 16 + (lane & 15);
          *reinterpret_cast<float*>(smem + r * kRowStride + (c >> 6) * kSegStride + (c & 63) * 4) =
              acc[mi][ni][i] * rs[mi][i];
        }
    __syncthreads();
    // scan 64 logits of row srow
    const uint8_t* base = smem + srow * kRowStride + sseg * kSegStride;
    const int c0 = n0 + sseg * kSegCols;
#pragma unroll 4
    for (int c4 = 0; c4 < kSegCols; c4 += 4) {
      const float4 v4 = *reinterpret_cast<const float4*>(base + c4 * 4);
      const float vv[4] = {v4.x, v4.y, v4.z, v4.w};
      bool ok[4];
      float cmax = -INFINITY;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int col = c0 + c4 + e;
        ok[e] = col < V && col != mask_id;
        if (ok[e]) cmax = fmaxf(cmax, vv[e]);
      }
      if (cmax > m) {  // rescale the running sums to the new max
        if (m > -INFINITY) {
          const float alpha = fast_exp(m - cmax);
          t = alpha * (t + (m - cmax) * s);
          s = alpha * s;
        }
        m = cmax;
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (!ok[e]) continue;
        const float x = vv[e] - m;
        const float ex = fast_exp(x);
        s += ex;
        t += ex * x;
        if (better(vv[e], c0 + c4 + e, tv[kK - 1], ti[kK - 1])) topk_insert(tv, ti, vv[e], c0 + c4 + e);
      }
    }
    __syncthreads();
  }
  const int row = m0 + srow;
  if (row < R) {
    const size_t p = size_t(row) * part.P + size_t(slice) * kSegs + sseg;
    part.m[p] = m;
    part.s[p] = s;
    part.t[p] = t;
#pragma unroll
    for (int k = 0; k < kK; ++k) {
      part.tv[p * kK + k] = tv[k];
      part.ti[p * kK + k] = ti[k];
    }
  }
}

// One wave per row.
__global__ __launch_bounds__(256) void merge_kernel(Partials part, int R, StatsOut out) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= R) return;
  const size_t base = size_t(row) * part.P;
  float M = -INFINITY;
  for (int p = lane; p < part.P; p += 64) M = fmaxf(M, part.m[base + p]);
  M = wave_max(M);
  float S = 0.f, Tt = 0.f;
  float tv[kK];
  int ti[kK];
#pragma unroll
  for (int k = 0; k < kK; ++k) { tv[k] = -INFINITY; ti[k] = 0x7fffffff; }
  for (int p = lane; p < part.P; p += 64) {
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
  // 64-way merge of the lanes' sorted lists: the wave-wide best head is taken K times
  for (int k = 0; k < out.k; ++k) {
    float v = tv[0];
    int i = ti[0];
    wave_argmax(v, i);
    if (lane == 0) {
      out.topk_id[size_t(row) * out.k + k] = i;
      out.topk_logit[size_t(row) * out.k + k] = v;
    }
    if (ti[0] == i) {  // ids are unique: exactly one lane owns the winner; pop it
#pragma unroll
      for (int j = 0; j < kK - 1; ++j) { tv[j] = tv[j + 1]; ti[j] = ti[j + 1]; }
      tv[kK - 1] = -INFINITY;
      ti[kK - 1] = 0x7fffffff;
    }
    if (k == 0 && lane == 0) out.argmax[row] = i;
  }
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
  const int rt = cdiv(R, kRows), vt = cdiv(V, kCols);
  return std::max(1, std::min(vt, cdiv(kTargetWg, rt)));
}

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
  const size_t P = size_t(slices_for(R, V)) * kSegs;
  return size_t(R) * P * (3 + 2 * kK) * 4 + 256;
}

hipError_t lmhead_partials(int dtype, const void* h, const void* w, int R, int d, int V, const float* row_scale,
                           const int32_t* rs_idx, int rs_n, int rs_lim, float scale, int mask_id, void* ws,
                           hipStream_t s) {
  if (d <= 0 || d % (dtype ? 64 : 32)) return hipErrorInvalidValue;   // the mainloop runs stages in pairs
  const int ns = slices_for(R, V);
  const int rt = cdiv(R, kRows), vt = cdiv(V, kCols);
  Partials part = carve(ws, R, ns * kSegs);
  const int grid = rt * ns;
  if (dtype)
    hipLaunchKernelGGL(lmhead_kernel<bf16_t>, dim3(grid), dim3(kThreads), 0, s, static_cast<const bf16_t*>(h),
                       static_cast<const bf16_t*>(w), R, d, V, row_scale, rs_idx, rs_n, rs_lim, scale, mask_id, rt,
                       ns, vt, part);
  else
    hipLaunchKernelGGL(lmhead_kernel<float>, dim3(grid), dim3(kThreads), 0, s, static_cast<const float*>(h),
                       static_cast<const float*>(w), R, d, V, row_scale, rs_idx, rs_n, rs_lim, scale, mask_id, rt,
                       ns, vt, part);
  return hipGetLastError();
}

hipError_t lmhead_merge(int R, int V, const StatsOut& out, void* ws, hipStream_t s) {
  Partials part = carve(ws, R, slices_for(R, V) * kSegs);
  hipLaunchKernelGGL(merge_kernel, dim3(cdiv(R, 4)), dim3(256), 0, s, part, R, out);
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
