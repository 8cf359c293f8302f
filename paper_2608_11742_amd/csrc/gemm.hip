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
constexpr int kWavesM = 4, kWavesN = 2;   // 8 waves of 64 x 128, two per SIMD
using Tile = TileMma<bf16_t, kBM, kBN, kWavesM, kWavesN>;  // geometry is the same for fp32
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

// HD: head_dim of the QKV epilogue (compile-time, so the rotary partner block
// index stays static and the accumulators stay in registers); 0 otherwise.
template <typename T, int EPI, int HD>
__global__ __launch_bounds__(kThreads, 2) void gemm_kernel(const T* __restrict__ A, int lda,
                                                           const T* __restrict__ B, int ldb, int M, int N, int K,
                                                           int tiles_m, int tiles_n, EpiParams ep) {
  using TM = TileMma<T, kBM, kBN, kWavesM, kWavesN>;
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
  const int wm = wave / kWavesN, wn = wave % kWavesN;
  const int row_base = m0 + wm * TM::kWTM + 4 * (lane >> 4);
  const int lc = lane & 15;

  if constexpr (EPI == EPI_RESID) {
    // x += acc through LDS: each wave stages half of its 64 x 128 tile at a
    // time (64 x 64 fp32, 16 KB, in its own region of the idle ring), rows of
    // 16 chunks of 4 floats with chunk c of row r in slot c ^ (r % 16), so
    // both the MFMA-layout writes and the row reads are conflict-free; then
    // every lane reads 16 bytes of x per access, all loads first (clamped
    // into the matrix) and the guarded stores after them.
    static_assert(TM::kWTM == 64 && TM::kWTN == 128, "resid epilogue tiling");
    uint8_t* st = smem + wave * (64 * 64 * 4);
    auto slot_of = [](int r, int c4) { return r * 256 + (((c4 ^ (r & 15))) << 4); };
    const int r0 = m0 + wm * 64;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
#pragma unroll
      for (int m = 0; m < TM::kFM; ++m)
#pragma unroll
        for (int nn = 0; nn < 4; ++nn)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int r = m * 16 + 4 * (lane >> 4) + i, c = nn * 16 + lc;
            *reinterpret_cast<float*>(st + slot_of(r, c >> 2) + (c & 3) * 4) = acc[m][4 * h + nn][i];
          }
      const int c0 = tn * kBN + wn * TM::kWTN + 64 * h;
      f32x4 xv[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int q = lane + 64 * j, r = q >> 4, c4 = q & 15;
        const int row = min(r0 + r, M - 1), col = min(c0 + 4 * c4, N - 4);
        xv[j] = *reinterpret_cast<const f32x4*>(ep.x + size_t(row) * ep.ldx + col);
      }
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int q = lane + 64 * j, r = q >> 4, c4 = q & 15;
        const int row = r0 + r, col = c0 + 4 * c4;
        const f32x4 a = *reinterpret_cast<const f32x4*>(st + slot_of(r, c4));
        if (row < M && col < N) *reinterpret_cast<f32x4*>(ep.x + size_t(row) * ep.ldx + col) = xv[j] + a;
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
    static_assert(HD == 64 || HD == 128, "head_dim");
    const QkvOut& o = ep.qkv;
    constexpr int hd = HD, half = HD / 2, pair = HD / 32;  // partner block distance
    const int wcol0 = tn * kBN + wn * TM::kWTN;            // first column of this wave tile
    const int which = wcol0 / o.d;                         // 0: q, 1: k, 2: v (uniform per wave)
    const int cin0 = wcol0 % o.d;
    // rotary embedding in registers: (x1, x2) = columns (dim, dim + hd/2) of one head
    if (which < 2) {
#pragma unroll
      for (int m = 0; m < TM::kFM; ++m) {
        // one 16-row block at a time: keeps the cos/sin loads of all blocks
        // from being hoisted together into the registers
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = min(row_base + m * 16 + i, M - 1);
          const int r = row % o.seq;
          const int pos = o.pos_offset + (o.pack_B && r >= o.pack_S ? o.pack_b0 + ((r - o.pack_S) & (o.pack_B - 1)) : r);
#pragma unroll
          for (int n = 0; n < TM::kFN; ++n) {
            if constexpr (true) {
              if (((n * 16) % hd) >= half) continue;
              const int dim = (cin0 + n * 16 + lc) % hd;
              const float2 cs = o.rope[size_t(pos) * half + dim];
              const float x1 = acc[m][n][i], x2 = acc[m][n + pair][i];
              acc[m][n][i] = x1 * cs.x - x2 * cs.y;
              acc[m][n + pair][i] = x1 * cs.y + x2 * cs.x;
            }
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (Elem<T>::bytes == 2) {
      // stage the wave's 64 x 128 tile as bf16 in LDS (V transposed), then write
      // 16-byte chunks: Q/K rows are contiguous along head_dim, V^T rows along positions
      uint8_t* st = smem + wave * (TM::kWTM * TM::kWTN * 2);
      if (which < 2) {
#pragma unroll
        for (int m = 0; m < TM::kFM; ++m)
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int n = 0; n < TM::kFN; ++n) {
              const int r = m * 16 + 4 * (lane >> 4) + i, c = n * 16 + lc;
              *reinterpret_cast<uint16_t*>(st + (r * TM::kWTN + c) * 2) = f2bf(acc[m][n][i]);
            }
      } else {
#pragma unroll
        for (int m = 0; m < TM::kFM; ++m)
#pragma unroll
          for (int n = 0; n < TM::kFN; ++n) {
            const int r = m * 16 + 4 * (lane >> 4), c = n * 16 + lc;
            const uint32_t lo = uint32_t(f2bf(acc[m][n][0])) | (uint32_t(f2bf(acc[m][n][1])) << 16);
            const uint32_t hi = uint32_t(f2bf(acc[m][n][2])) | (uint32_t(f2bf(acc[m][n][3])) << 16);
            *reinterpret_cast<u32x2*>(st + (c * TM::kWTM + r) * 2) = u32x2{lo, hi};
          }
      }
      __syncthreads();
      const int r0 = m0 + wm * TM::kWTM;
      if (which < 2) {
        uint16_t* dst = reinterpret_cast<uint16_t*>(which == 0 ? o.q : o.k);
        for (int q = lane; q < TM::kWTM * TM::kWTN / 8; q += 64) {
          const int r = q / (TM::kWTN / 8), c8 = (q % (TM::kWTN / 8)) * 8;
          const int row = r0 + r;
          if (row >= M) continue;
          const int b = row / o.seq, sp = row % o.seq;
          const int cin = cin0 + c8, h = cin / hd, dim = cin % hd;
          *reinterpret_cast<u32x4*>(dst + (size_t(b * o.H + h) * o.seq + sp) * hd + dim) =
              *reinterpret_cast<const u32x4*>(st + (r * TM::kWTN + c8) * 2);
        }
      } else {
        uint16_t* dst = reinterpret_cast<uint16_t*>(o.vt);
        const bool aligned = (o.seq % 8) == 0;
        for (int q = lane; q < TM::kWTM * TM::kWTN / 8; q += 64) {
          const int c = q / (TM::kWTM / 8), rr = (q % (TM::kWTM / 8)) * 8;
          const int cin = cin0 + c, h = cin / hd, dim = cin % hd;
          const int row = r0 + rr;
          if (row >= M) continue;
          if (aligned && row + 7 < M) {
            const int b = row / o.seq, sp = row % o.seq;
            *reinterpret_cast<u32x4*>(dst + (size_t(b * o.H + h) * hd + dim) * o.vt_ld + sp) =
                *reinterpret_cast<const u32x4*>(st + (c * TM::kWTM + rr) * 2);
          } else {
            for (int e = 0; e < 8 && row + e < M; ++e) {
              const int b = (row + e) / o.seq, sp = (row + e) % o.seq;
              dst[(size_t(b * o.H + h) * hd + dim) * o.vt_ld + sp] =
                  *reinterpret_cast<const uint16_t*>(st + (c * TM::kWTM + rr + e) * 2);
            }
          }
        }
      }
    } else {
      // fp32 activations: direct element stores
#pragma unroll
      for (int m = 0; m < TM::kFM; ++m)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = row_base + m * 16 + i;
          if (row >= M) continue;
          const int b = row / o.seq, sp = row % o.seq;
#pragma unroll
          for (int n = 0; n < TM::kFN; ++n) {
            const int cin = cin0 + n * 16 + lc;
            const int h = cin / hd, dim = cin % hd;
            T* dst = which == 2 ? reinterpret_cast<T*>(o.vt) + (size_t(b * o.H + h) * hd + dim) * o.vt_ld + sp
                                : reinterpret_cast<T*>(which == 0 ? o.q : o.k) + (size_t(b * o.H + h) * o.seq + sp) * hd +
                                      dim;
            store_f(dst, acc[m][n][i]);
          }
        }
    }
  }
}

template <typename T, int EPI, int HD = 0>
hipError_t launch(const void* A, int lda, const void* B, int ldb, int M, int N, int K, int tiles_n,
                  const EpiParams& ep, hipStream_t s) {
  // the mainloop runs stages in pairs
  if (K <= 0 || K % (2 * TileMma<T, kBM, kBN, kWavesM, kWavesN>::kKPerStage)) return hipErrorInvalidValue;
  const int tiles_m = cdiv(M, kBM);
  const int grid = tiles_m * tiles_n;
  hipLaunchKernelGGL((gemm_kernel<T, EPI, HD>), dim3(grid), dim3(kThreads), 0, s, static_cast<const T*>(A), lda,
                     static_cast<const T*>(B), ldb, M, N, K, tiles_m, tiles_n, ep);
  return hipGetLastError();
}

}  // namespace

hipError_t gemm_resid(int dtype, const void* A, int lda, const void* B, int ldb, int M, int N, int K, float* X,
                      int ldx, hipStream_t s) {
  if (N % 4 || ldx % 4 || reinterpret_cast<uintptr_t>(X) % 16) return hipErrorInvalidValue;   // 16-byte x accesses
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
  if (o.hd == 128)
    return dtype ? launch<bf16_t, EPI_QKV, 128>(A, lda, Wqkv, K, M, N, K, tn, ep, s)
                 : launch<float, EPI_QKV, 128>(A, lda, Wqkv, K, M, N, K, tn, ep, s);
  return dtype ? launch<bf16_t, EPI_QKV, 64>(A, lda, Wqkv, K, M, N, K, tn, ep, s)
               : launch<float, EPI_QKV, 64>(A, lda, Wqkv, K, M, N, K, tn, ep, s);
}

}  // namespace dllm
