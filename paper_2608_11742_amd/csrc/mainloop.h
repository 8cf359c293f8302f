// Block-tile MFMA mainloop for C = A B^T with A [M][K] and B [N][K] both
// K-contiguous (the [out][in] weight layout), fp32 accumulation.
//
// A workgroup computes a BM x BN tile with WAVES_M x WAVES_N waves; each wave
// owns a (BM/WAVES_M) x (BN/WAVES_N) sub-tile made of 16x16 MFMA blocks.
// K advances in stages of 128 bytes per row (64 bf16 or 32 fp32 values):
// every thread fetches its share of the next stage into registers while the
// waves multiply the current stage out of LDS, then writes it to the other of
// two LDS buffers (one barrier per stage).  LDS rows are 8 chunks of 16
// bytes; chunk c of row r lives at chunk slot c ^ (r & 7), so the 16-byte
// fragment reads of 8 consecutive rows hit 8 different bank groups.
#pragma once

#include "common.h"

namespace dllm {

template <typename T, int BM, int BN, int WAVES_M, int WAVES_N>
struct TileMma {
  static constexpr int kThreads = WAVES_M * WAVES_N * kWave;
  static constexpr int kWTM = BM / WAVES_M;
  static constexpr int kWTN = BN / WAVES_N;
  static constexpr int kFM = kWTM / 16;
  static constexpr int kFN = kWTN / 16;
  static constexpr int kRowBytes = 128;
  static constexpr int kStageA = BM * kRowBytes;
  static constexpr int kStageB = BN * kRowBytes;
  static constexpr int kStage = kStageA + kStageB;
  static constexpr int kSmem = 2 * kStage;
  static constexpr int kACh = BM * 8 / kThreads;   // A chunks per thread per stage
  static constexpr int kBCh = BN * 8 / kThreads;
  static constexpr int kKPerStage = kRowBytes / Elem<T>::bytes;
  static_assert(kACh * kThreads == BM * 8 && kBCh * kThreads == BN * 8, "tile / thread mismatch");
  static_assert(kWTM % 16 == 0 && kWTN % 16 == 0, "wave tile must be 16-aligned");

  __device__ __forceinline__ static int swz(int r, int c) { return r * kRowBytes + ((c ^ (r & 7)) << 4); }

  // a_off(r) / b_off(r): byte offset of local row r (already clamped to a
  // valid row) relative to A / B.  nk: number of K stages.
  template <class AOff, class BOff>
  __device__ __forceinline__ static void run(uint8_t* smem, const uint8_t* A, const uint8_t* B, AOff a_off,
                                             BOff b_off, int nk, f32x4 (&acc)[kFM][kFN]) {
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WAVES_N;
    const int wn = wave % WAVES_N;

    uint32_t ga[kACh], gb[kBCh];
    int sa[kACh], sb[kBCh];
#pragma unroll
    for (int i = 0; i < kACh; ++i) {
      int q = tid + kThreads * i, r = q >> 3, c = q & 7;
      ga[i] = a_off(r) + c * 16;
      sa[i] = swz(r, c);
    }
#pragma unroll
    for (int i = 0; i < kBCh; ++i) {
      int q = tid + kThreads * i, r = q >> 3, c = q & 7;
      gb[i] = b_off(r) + c * 16;
      sb[i] = kStageA + swz(r, c);
    }
#pragma unroll
    for (int m = 0; m < kFM; ++m)
#pragma unroll
      for (int n = 0; n < kFN; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};

    u32x4 ra[kACh], rb[kBCh];
    auto gload = [&](int kt) {
      const uint32_t koff = uint32_t(kt) * kRowBytes;
#pragma unroll
      for (int i = 0; i < kACh; ++i) ra[i] = *reinterpret_cast<const u32x4*>(A + ga[i] + koff);
#pragma unroll
      for (int i = 0; i < kBCh; ++i) rb[i] = *reinterpret_cast<const u32x4*>(B + gb[i] + koff);
    };
    auto sstore = [&](int buf) {
      uint8_t* s = smem + buf * kStage;
#pragma unroll
      for (int i = 0; i < kACh; ++i) *reinterpret_cast<u32x4*>(s + sa[i]) = ra[i];
#pragma unroll
      for (int i = 0; i < kBCh; ++i) *reinterpret_cast<u32x4*>(s + sb[i]) = rb[i];
    };

    // fragment read offsets: lane reads row (block row + lane % 16), chunk 4*step + lane / 16
    const int fr = lane & 15;
    const int fc = lane >> 4;

    gload(0);
    sstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      if (kt + 1 < nk) gload(kt + 1);
      const uint8_t* s = smem + (kt & 1) * kStage;
#pragma unroll
      for (int step = 0; step < 2; ++step) {
        u32x4 af[kFM], bfr[kFN];
#pragma unroll
        for (int m = 0; m < kFM; ++m)
          af[m] = *reinterpret_cast<const u32x4*>(s + swz(wm * kWTM + m * 16 + fr, 4 * step + fc));
#pragma unroll
        for (int n = 0; n < kFN; ++n)
          bfr[n] = *reinterpret_cast<const u32x4*>(s + kStageA + swz(wn * kWTN + n * 16 + fr, 4 * step + fc));
#pragma unroll
        for (int m = 0; m < kFM; ++m)
#pragma unroll
          for (int n = 0; n < kFN; ++n) Mfma<T>::run(acc[m][n], af[m], bfr[n]);
      }
      if (kt + 1 < nk) sstore((kt + 1) & 1);
      __syncthreads();
    }
  }
};

// Map a linear workgroup id to a (tile_m, tile_n) pair.  Workgroups are
// dispatched round-robin over the 8 XCDs, each with its own L2; the id is
// first remapped so that every XCD receives a contiguous range, then tiles
// are walked in groups of `group_m` row-tiles so that neighbours share A and
// B tiles in that XCD's L2.
__device__ __forceinline__ void map_tile(int id, int nwg, int tiles_m, int tiles_n, int group_m, int& tm,
                                         int& tn) {
  const int q = nwg / 8, r = nwg % 8;
  const int xcd = id % 8, local = id / 8;
  const int lin = xcd < r ? xcd * (q + 1) + local : r * (q + 1) + (xcd - r) * q + local;
  const int group = group_m * tiles_n;
  const int g = lin / group;
  const int first_m = g * group_m;
  const int gm = min(tiles_m - first_m, group_m);
  const int in_g = lin % group;
  tm = first_m + in_g % gm;
  tn = in_g / gm;
}

}  // namespace dllm
