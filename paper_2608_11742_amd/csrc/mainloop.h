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
// LDS layout of a stage: rows are paired into 128-byte lines, row r in line
// r / 2; a line holds 8 chunks of 16 bytes, and logical chunk c of row r
// (position (r % 2) * 4 + c in its line) sits in slot position ^ (line % 8).
// A fragment read (16 consecutive rows at one chunk per 16 lanes) then runs
// at the full LDS read rate of gfx950; plain or row-XOR-swizzled 64-byte rows
// measure at half of it.  A load-to-LDS instruction writes 64 lanes x 16
// bytes contiguously (8 lines = 16 rows); lane l fills line l / 8, slot l % 8,
// and so fetches the row and chunk that the swizzle assigns to that slot.
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

// s_waitcnt lgkmcnt(0) (vmcnt and expcnt left unconstrained)
__device__ __forceinline__ void wait_lgkmcnt0() { __builtin_amdgcn_s_waitcnt((0xF) | (0x3 << 14) | (0x7 << 4)); }

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

  // byte offset within a stage of logical chunk c (0..3) of local row r
  __device__ __forceinline__ static int swz(int r, int c) {
    const int line = r >> 1;
    return line * 128 + (((((r & 1) << 2) | c) ^ (line & 7)) << 4);
  }
  // (row, chunk) that lane l of load instruction `grp` (rows 16 grp .. 16 grp + 15) fetches
  __device__ __forceinline__ static int dma_row(int grp, int l) {
    const int q = l >> 3, s = (l & 7) ^ q;
    return grp * 16 + 2 * q + (s >> 2);
  }
  __device__ __forceinline__ static int dma_chunk(int l) { return ((l & 7) ^ (l >> 3)) & 3; }

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
    for (int i = 0; i < kIA; ++i) ga[i] = a_off(dma_row(wave * kIA + i, lane)) + (dma_chunk(lane) << 4);
#pragma unroll
    for (int i = 0; i < kIB; ++i) gb[i] = b_off(dma_row(wave * kIB + i, lane)) + (dma_chunk(lane) << 4);
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

    // Every step has the same shape: no branch but the loop's back-edge (a
    // branch inside a step makes the compiler's wait-count analysis wait for
    // the next stage's fragment reads before the MFMAs of the current one).
    // Past the last stage the loads repeat stage nk - 1 into the free ring
    // buffer, so that the number of loads in flight, and with it every vmcnt
    // wait, stays uniform.  Such a buffer is never read as a live stage: at
    // step kt it is the buffer of stage kt - 1, and the at most NS - 2 stages
    // still to be read occupy the buffers of kt + 1 .. kt + NS - 2.
#pragma unroll
    for (int s = 0; s < NS - 1; ++s) issue(min(s, nk - 1), s);
    wait_vmcnt<(NS - 2) * (kIA + kIB)>();   // stage 0 landed
    __syncthreads();
    read_frags(0, 0);
    // Step kt multiplies stage kt (fragments already in registers) while the
    // fragments of stage kt + 1 are read.  Its barrier needs stage kt + 1
    // landed in every wave; it also proves every wave has finished reading
    // stage kt - 1 (read during step kt - 2), so that buffer takes the load
    // of stage kt + NS - 1.  nk is even (checked by the launchers).
    // Scheduling fences keep each step's fragment reads ahead of its MFMAs
    // and the MFMAs inside their step; left free, the scheduler pairs every
    // read with the MFMA that consumes it and undoes the pipelining.
    auto step = [&](int kt, auto cur, auto nxt) {
      __builtin_amdgcn_sched_barrier(0);
      wait_vmcnt<kInflightNext>();
      __syncthreads();
      issue(min(kt + NS - 1, nk - 1), (kt + NS - 1) % NS);
      read_frags(kt + 1, decltype(nxt)::value);
      __builtin_amdgcn_sched_barrier(0);
      mma(decltype(cur)::value);
    };
    using S0 = std::integral_constant<int, 0>;
    using S1 = std::integral_constant<int, 1>;
    for (int kt = 0; kt < nk; kt += 2) {
      step(kt, S0{}, S1{});
      step(kt + 1, S1{}, S0{});
    }
    wait_vmcnt<0>();
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
