// Projection GEMMs of the transformer layer with fused epilogues:
//   resid  : x += a W^T                      (O and down projections)
//   swiglu : f = silu(a Wg^T) * (a Wu^T)     (gate/up projection)
//   qkv    : q, k, v = a Wqkv^T, rotary embedding on q and k, scattered to
//            head-major Q/K and transposed V
// 256x256 output tiles, 8 waves of 64x128, bf16 (or fp32) MFMA, fp32 accumulate.
#include "kernels.h"
#include "mainloop.h"

namespace dllm {

namespace {

constexpr int kBM = 256, kBN = 256;
using Tile = TileMma<bf16_t, kBM, kBN, 4, 2>;  // geometry is the same for fp32
constexpr int kThreads = Tile::kThreads;
constexpr int kGroupM = 8;

enum { EPI_RESID = 0, EPI_SWIGLU = 1, EPI_QKV = 2 };

struct EpiParams {
  float* x;          // resid: fp32 residual
  int ldx;
  void* out;         // swiglu: [M][F]
  int F;
  QkvOut qkv;
};

template <typename T, int EPI>
__global__ __launch_bounds__(kThreads, 2) void gemm_kernel(const T* __restrict__ A, int lda,
                                                           const T* __restrict__ B, int ldb, int M, int N, int K,
                                                           int tiles_m, int tiles_n, EpiParams ep) {
  using TM = TileMma<T, kBM, kBN, 4, 2>;
  __shared__ __attribute__((aligned(16))) uint8_t smem[TM::kSmem];
  int tm, tn;
  map_tile(blockIdx.x, gridDim.x, tiles_m, tiles_n, kGroupM, tm, tn);
  const int m0 = tm * kBM;
  const uint32_t a_row_bytes = uint32_t(lda) * sizeof(T);
  const uint32_t b_row_bytes = uint32_t(ldb) * sizeof(T);
  auto a_off = [&](int r) -> uint32_t { return uint32_t(min(m0 + r, M - 1)) * a_row_bytes; };
  auto b_off = [&](int r) -> uint32_t {
    int row;
    if constexpr (EPI == EPI_SWIGLU) {
      // 256 B rows -> 128 outputs: each 128-row half of a wave column pairs 64 gate and 64 up rows
      const int wn = r >> 7, rr = r & 127;
      const int j = min(tn * 128 + wn * 64 + (rr & 63), ep.F - 1);
      row = rr < 64 ? j : ep.F + j;
    } else {
      row = min(tn * kBN + r, N - 1);
    }
    return uint32_t(row) * b_row_bytes;
  };
  f32x4 acc[TM::kFM][TM::kFN];
  TM::run(smem, reinterpret_cast<const uint8_t*>(A), reinterpret_cast<const uint8_t*>(B), a_off, b_off,
          K / TM::kKPerStage, acc);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / 2, wn = wave % 2;
  const int row_base = m0 + wm * TM::kWTM + 4 * (lane >> 4);
  const int lc = lane & 15;

  if constexpr (EPI == EPI_RESID) {
    const int col_base = tn * kBN + wn * TM::kWTN + lc;
#pragma unroll
    for (int m = 0; m < TM::kFM; ++m)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = row_base + m * 16 + i;
        if (row >= M) continue;
        float* xr = ep.x + size_t(row) * ep.ldx;
#pragma unroll
        for (int n = 0; n < TM::kFN; ++n) {
          const int col = col_base + n * 16;
          if (col < N) xr[col] += acc[m][n][i];
        }
      }
  } else if constexpr (EPI == EPI_SWIGLU) {
    T* out = reinterpret_cast<T*>(ep.out);
#pragma unroll
    for (int m = 0; m < TM::kFM; ++m)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = row_base + m * 16 + i;
        if (row >= M) continue;
#pragma unroll
        for (int n = 0; n < TM::kFN / 2; ++n) {
          const int j = tn * 128 + wn * 64 + n * 16 + lc;
          if (j >= ep.F) continue;
          const float g = acc[m][n][i], u = acc[m][n + TM::kFN / 2][i];
          const float silu = g / (1.0f + __expf(-g));
          store_f(out + size_t(row) * ep.F + j, silu * u);
        }
      }
  } else {  // EPI_QKV
    const QkvOut& o = ep.qkv;
    const int hd = o.hd, half = hd / 2, pair = hd / 32;  // partner block distance
    const int wcol0 = tn * kBN + wn * TM::kWTN;            // first column of this wave tile
    if (wcol0 >= N) return;
    const int which = wcol0 / o.d;                         // 0: q, 1: k, 2: v
    const int cin0 = wcol0 % o.d;
#pragma unroll
    for (int m = 0; m < TM::kFM; ++m)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = row_base + m * 16 + i;
        if (row >= M) continue;
        const int b = row / o.seq, s = row % o.seq;
        const int pos = o.pos_offset + s;
#pragma unroll
        for (int n = 0; n < TM::kFN; ++n) {
          const int cin = cin0 + n * 16 + lc;
          const int h = cin / hd, dim = cin % hd;
          const float x1 = acc[m][n][i];
          if (which == 2) {
            T* vt = reinterpret_cast<T*>(o.vt);
            store_f(vt + (size_t(b * o.H + h) * hd + dim) * o.vt_ld + s, x1);
            continue;
          }
          if (((n * 16) % hd) >= half) continue;           // second half: written with its partner
          float x2 = 0.f;
#pragma unroll
          for (int p = 0; p < TM::kFN; ++p)
            if (p == n + pair) x2 = acc[m][p][i];
          const float2 cs = o.rope[size_t(pos) * half + dim];
          T* dst = reinterpret_cast<T*>(which == 0 ? o.q : o.k) + (size_t(b * o.H + h) * o.seq + s) * hd;
          store_f(dst + dim, x1 * cs.x - x2 * cs.y);
          store_f(dst + dim + half, x1 * cs.y + x2 * cs.x);
        }
      }
  }
}

template <typename T, int EPI>
hipError_t launch(const void* A, int lda, const void* B, int ldb, int M, int N, int K, int tiles_n,
                  const EpiParams& ep, hipStream_t s) {
  const int tiles_m = cdiv(M, kBM);
  const int grid = tiles_m * tiles_n;
  hipLaunchKernelGGL((gemm_kernel<T, EPI>), dim3(grid), dim3(kThreads), 0, s, static_cast<const T*>(A), lda,
                     static_cast<const T*>(B), ldb, M, N, K, tiles_m, tiles_n, ep);
  return hipGetLastError();
}

}  // namespace

hipError_t gemm_resid(int dtype, const void* A, int lda, const void* B, int ldb, int M, int N, int K, float* X,
                      int ldx, hipStream_t s) {
  EpiParams ep{};
  ep.x = X;
  ep.ldx = ldx;
  const int tn = cdiv(N, kBN);
  return dtype ? launch<bf16_t, EPI_RESID>(A, lda, B, ldb, M, N, K, tn, ep, s)
               : launch<float, EPI_RESID>(A, lda, B, ldb, M, N, K, tn, ep, s);
}

hipError_t gemm_swiglu(int dtype, const void* A, int lda, const void* Wgu, int M, int F, int K, void* out,
                       hipStream_t s) {
  EpiParams ep{};
  ep.out = out;
  ep.F = F;
  const int tn = cdiv(F, 128);
  return dtype ? launch<bf16_t, EPI_SWIGLU>(A, lda, Wgu, K, M, 2 * F, K, tn, ep, s)
               : launch<float, EPI_SWIGLU>(A, lda, Wgu, K, M, 2 * F, K, tn, ep, s);
}

hipError_t gemm_qkv(int dtype, const void* A, int lda, const void* Wqkv, int M, int K, const QkvOut& o,
                    hipStream_t s) {
  EpiParams ep{};
  ep.qkv = o;
  const int N = 3 * o.d;
  const int tn = cdiv(N, kBN);
  return dtype ? launch<bf16_t, EPI_QKV>(A, lda, Wqkv, K, M, N, K, tn, ep, s)
               : launch<float, EPI_QKV>(A, lda, Wqkv, K, M, N, K, tn, ep, s);
}

}  // namespace dllm
