// Block-tile MFMA mainloop for C = A B^T with A [M][K] and B [N][K] both
// K-contiguous (the [out][in] weight layout), fp32 accumulation.
//
// A workgroup computes a BM x BN tile with WAVES_M x WAVES_N waves; each wave
// owns a (BM/WAVES_M) x (BN/WAVES_N) sub-tile made of 16x16 MFMA blocks.
// K advances in stages of 64 bytes per row (32 bf16 or 16 fp32 values).
// Stages are copied from global memory straight into a ring of NS LDS
// buffers with global_load_lds_dwordx4 (no register staging), NS - 1 stages
// ahead of the stage being multiplied, so a load has NS - 2 stages of MFMA
// work to land; the MMA fragments of the next stage are read from LDS while
// the current stage's MFMAs run; one barrier per stage.
//
// LDS layout of a stage: row r is 4 chunks of 16 bytes; logical chunk c of
// row r sits in slot c ^ perm(r), so the 16-byte fragment reads of
// consecutive rows at the same logical chunk hit distinct banks.  A
// load-to-LDS instruction writes 64 lanes x 16 bytes contiguously (16 rows);
// lane l therefore fetches row l / 4 of its group at the logical chunk that
// belongs in slot l % 4.
#pragma once

#include <type_traits>

#include "common.h"

namespace dllm {

// Asynchronous 16-byte copy global -> LDS.  lds_addr is the wave-uniform LDS
// byte address of the 1 KB block the 64 lanes fill.  Issued through inline
// assembly so the compiler does not insert a conservative wait for it before
// every LDS read; completion is awaited explicitly with wait_vmcnt.
__device__ __forceinline__ void lds_dma16(const void* gptr, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(gptr), "s"(lds_addr) : "memory", "m0");
}

// s_waitcnt vmcnt(N) (expcnt and lgkmcnt left unconstrained)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | (((N >> 4) & 3) << 14) | (0x7 << 4) | (0xF << 8));
}

__device__ __forceinline__ uint32_t lds_address(const void* p) {
  // a generic pointer into LDS converted to the 32-bit LDS byte address
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) uint8_t*)(p)));
}

template <typename T, int BM, int BN, int WAVES_M, int WAVES_N, int NS = 4>
struct TileMma {
  static constexpr int kWaves = WAVES_M * WAVES_N;
  static constexpr int kThreads = kWaves * kWave;
  static constexpr int kWTM = BM / WAVES_M;
  static constexpr int kWTN = BN / WAVES_N;
  static constexpr int kFM = kWTM / 16;
  static constexpr int kFN = kWTN / 16;
  static constexpr int kRowBytes = 64;
  static constexpr int kStageA = BM * kRowBytes;
  static constexpr int kStageB = BN * kRowBytes;
  static constexpr int kStage = kStageA + kStageB;
  static constexpr int kSmem = NS * kStage;
  static constexpr int kKPerStage = kRowBytes / Elem<T>::bytes;
  static constexpr int kIA = BM / 16 / kWaves;   // load-to-LDS instructions per wave per stage (A)
  static constexpr int kIB = BN / 16 / kWaves;   // (B)
  // load instructions of later stages allowed in flight while stage kt + 1 must have landed
  static constexpr int kInflightNext = (NS - 3) * (kIA + kIB);
  static_assert(kIA * kWaves * 16 == BM && kIB * kWaves * 16 == BN, "tile / wave mismatch");
  static_assert(kWTM % 16 == 0 && kWTN % 16 == 0, "wave tile must be 16-aligned");
  static_assert(NS >= 3, "ring depth");

  // chunk slot permutation of row r: the 16-byte reads of 16 consecutive rows
  // at one logical chunk fall in 16 distinct 16-byte bank groups (and any 8
  // consecutive rows in 8 distinct groups of a 128-byte window)
  __device__ __forceinline__ static int perm(int r) { return ((r >> 1) ^ (r >> 3)) & 3; }
  __device__ __forceinline__ static int swz(int r, int c) { return r * kRowBytes + ((c ^ perm(r)) << 4); }

  // a_off(r) / b_off(r): byte offset of local row r (already clamped to a
  // valid row) relative to A / B.  nk: number of K stages.  smem: kSmem bytes.
  template <class AOff, class BOff>
  __device__ __forceinline__ static void run(uint8_t* smem, const uint8_t* A, const uint8_t* B, AOff a_off,
                                             BOff b_off, int nk, f32x4 (&acc)[kFM][kFN]) {
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WAVES_N;
    const int wn = wave % WAVES_N;

    // this lane's source rows/chunks for the wave's load instructions
    uint32_t ga[kIA], gb[kIB];
#pragma unroll
    for (int i = 0; i < kIA; ++i) {
      const int r = (wave * kIA + i) * 16 + (lane >> 2);
      ga[i] = a_off(r) + (((lane & 3) ^ perm(r)) << 4);
    }
#pragma unroll
    for (int i = 0; i < kIB; ++i) {
      const int r = (wave * kIB + i) * 16 + (lane >> 2);
      gb[i] = b_off(r) + (((lane & 3) ^ perm(r)) << 4);
    }
    const uint32_t lds0 = lds_address(smem);
    auto issue = [&](int kt, int buf) {
      const uint32_t koff = uint32_t(kt) * kRowBytes;
      const uint32_t sbase = lds0 + buf * kStage;
#pragma unroll
      for (int i = 0; i < kIA; ++i)
        lds_dma16(A + ga[i] + koff, __builtin_amdgcn_readfirstlane(sbase + (wave * kIA + i) * 1024));
#pragma unroll
      for (int i = 0; i < kIB; ++i)
        lds_dma16(B + gb[i] + koff, __builtin_amdgcn_readfirstlane(sbase + kStageA + (wave * kIB + i) * 1024));
    };

#pragma unroll
    for (int m = 0; m < kFM; ++m)
#pragma unroll
      for (int n = 0; n < kFN; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int fr = lane & 15;
    const int fc = lane >> 4;
    u32x4 af[2][kFM], bfr[2][kFN];   // fragments of the current and the next stage
    auto read_frags = [&](int kt, int slot) {
      const uint8_t* s = smem + (kt % NS) * kStage;
#pragma unroll
      for (int m = 0; m < kFM; ++m)
        af[slot][m] = *reinterpret_cast<const u32x4*>(s + swz(wm * kWTM + m * 16 + fr, fc));
#pragma unroll
      for (int n = 0; n < kFN; ++n)
        bfr[slot][n] = *reinterpret_cast<const u32x4*>(s + kStageA + swz(wn * kWTN + n * 16 + fr, fc));
    };
    auto mma = [&](int slot) {
#pragma unroll
      for (int m = 0; m < kFM; ++m)
#pragma unroll
        for (int n = 0; n < kFN; ++n) Mfma<T>::run(acc[m][n], af[slot][m], bfr[slot][n]);
    };

#pragma unroll
    for (int s = 0; s < NS - 1; ++s)
      if (s < nk) issue(s, s);
    wait_vmcnt<0>();
    __syncthreads();
    read_frags(0, 0);
    // Iteration kt multiplies stage kt (fragments already in registers) while
    // the fragments of stage kt + 1 are read.  Its barrier needs stage kt + 1
    // landed in every wave; it also proves every wave has finished reading
    // stage kt - 1 (read during iteration kt - 2), so that buffer takes the
    // load of stage kt + NS - 1.
    auto step = [&](int kt, auto cur, auto nxt) {
      if (kt + 1 < nk) {
        if (kt + NS - 2 < nk)
          wait_vmcnt<kInflightNext>();
        else
          wait_vmcnt<0>();
        __syncthreads();
        if (kt + NS - 1 < nk) issue(kt + NS - 1, (kt + NS - 1) % NS);
        read_frags(kt + 1, decltype(nxt)::value);
      }
      mma(decltype(cur)::value);
    };
    using S0 = std::integral_constant<int, 0>;
    using S1 = std::integral_constant<int, 1>;
    for (int kt = 0; kt < nk; kt += 2) {
      step(kt, S0{}, S1{});
      if (kt + 1 < nk) step(kt + 1, S1{}, S0{});
    }
    __syncthreads();   // the caller may reuse the LDS
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
