// Block-tile MFMA mainloop for C = A B^T with A [M][K] and B [N][K] both
// K-contiguous (the [out][in] weight layout), fp32 accumulation.
//
// A workgroup computes a BM x BN tile with WAVES_M x WAVES_N waves; each wave
// owns a (BM/WAVES_M) x (BN/WAVES_N) sub-tile made of 16x16 MFMA blocks.
// K advances in stages of 128 bytes per row (64 bf16 or 32 fp32 values),
// copied from global memory straight into a two-slot LDS ring with
// global_load_lds_dwordx4 (no register staging); each load instruction
// moves 8 whole 128-byte rows, i.e. full cache lines.  A stage is consumed
// in two MFMA sub-steps of 64 bytes of K; the fragments of the next
// sub-step are read from LDS while the current one's MFMAs run, and one
// barrier per stage hands the just-consumed slot to the load of the stage
// after next, so a load has a full stage of MFMA work to land.
//
// LDS layout of a stage: row r is 128 bytes = 8 chunks of 16 bytes, logical
// chunk c in slot c ^ (r % 8).  A fragment read (16 consecutive rows at one
// chunk per 16 lanes) then stays near the full LDS read rate of gfx950.  A
// load instruction writes 64 lanes x 16 bytes contiguously (8 rows); lane l
// fills row l / 8, slot l % 8, and so fetches the chunk that the swizzle
// assigns to that slot.
#pragma once

#include <type_traits>

#include "common.h"

namespace dllm {

// Buffer resource for a range starting at p (stride 0, 32-bit data format):
// num_records is the maximum, every offset used with it is a clamped
// in-range row offset.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
__device__ __forceinline__ rsrc_t buffer_rsrc(const void* p) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), /*stride=*/0, /*num_records=*/-1,
                                           /*flags=*/0x00020000);
}

// Asynchronous 16-byte-per-lane copy buffer -> LDS: lane l reads base +
// voff + soff and writes LDS byte lds_addr + 16 l, where lds_addr is the
// wave-uniform LDS address of the 1 KB block the 64 lanes fill.  The
// compiler's buffer-load-to-LDS builtin: it sets up M0 itself.  Completion
// is awaited explicitly with wait_vmcnt before the barrier that publishes a
// stage; the compiler does not wait for these copies before LDS reads.
__device__ __forceinline__ void lds_dma16(rsrc_t rsrc, uint32_t voff, uint32_t soff, uint32_t lds_addr) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(
      rsrc, reinterpret_cast<__attribute__((address_space(3))) void*>(static_cast<uintptr_t>(lds_addr)), 16, voff,
      soff, 0, 0);
}

// s_waitcnt vmcnt(N) (expcnt and lgkmcnt left unconstrained)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | (((N >> 4) & 3) << 14) | (0x7 << 4) | (0xF << 8));
}

// s_waitcnt lgkmcnt(0) (vmcnt and expcnt left unconstrained)
__device__ __forceinline__ void wait_lgkmcnt0() { __builtin_amdgcn_s_waitcnt((0xF) | (0x3 << 14) | (0x7 << 4)); }

// Workgroup barrier after this wave's LDS operations have completed, without
// waiting for its outstanding copies into LDS (the workgroup fence of
// __syncthreads would wait for those too).  The signal fences keep the
// compiler from moving memory accesses across it.
__device__ __forceinline__ void barrier_lds() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  wait_lgkmcnt0();
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// f(integral_constant<int, i>) for i = B .. E - 1, unrolled at compile time
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

__device__ __forceinline__ uint32_t lds_address(const void* p) {
  // a generic pointer into LDS converted to the 32-bit LDS byte address
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) uint8_t*)(p)));
}

// TRANS: every 16x16 block is computed as (B A^T)^T, so that lane l holds
// row 16 m + l % 16 and the 4 consecutive columns 16 n + 4 (l / 16) + i of
// block (m, n) (instead of 4 consecutive rows of one column): row-contiguous
// epilogues then store 4 values per lane.
//
// EARLY: two barriers per stage instead of one.  The first follows sub-step
// 0, once every wave has read its last fragments of the stage, and hands the
// slot to the copies of stage j + 2 at once; the second, later in sub-step 1,
// publishes stage j + 1.  A copy then has about 1.2-1.3 stages of MFMA work to
// land instead of 0.65-1.0, for launches whose operands stream from HBM with
// too few bytes in flight per CU to cover its latency.
template <typename T, int BM, int BN, int WAVES_M, int WAVES_N, bool TRANS = false, bool EARLY = false>
struct TileMma {
  static constexpr int kWaves = WAVES_M * WAVES_N;
  static constexpr int kThreads = kWaves * kWave;
  static constexpr int kWTM = BM / WAVES_M;
  static constexpr int kWTN = BN / WAVES_N;
  static constexpr int kFM = kWTM / 16;
  static constexpr int kFN = kWTN / 16;
  static constexpr int kRowBytes = 128;                    // one stage of one row
  static constexpr int kStageA = BM * kRowBytes;
  static constexpr int kStageB = BN * kRowBytes;
  static constexpr int kStage = kStageA + kStageB;
  static constexpr int kSmem = 2 * kStage;
  static constexpr int kKPerStage = 64 / Elem<T>::bytes;   // K of one MFMA sub-step; K must be a multiple of twice this
  static constexpr int kIA = BM / 8 / kWaves;               // load-to-LDS instructions per wave per stage (A)
  static constexpr int kIB = BN / 8 / kWaves;               // (B)
  static_assert(kIA * kWaves * 8 == BM && kIB * kWaves * 8 == BN, "tile / wave mismatch");
  static_assert(kWTM % 16 == 0 && kWTN % 16 == 0, "wave tile must be 16-aligned");

  // byte offset within a stage of logical chunk c (0..7) of local row r
  __device__ __forceinline__ static int swz(int r, int c) { return r * kRowBytes + ((c ^ (r & 7)) << 4); }

  // The wave's share of the global -> LDS copies of one tile: lane source
  // offsets and buffer descriptors.  a_off(r) / b_off(r): byte offset of
  // local row r (already clamped to a valid row) relative to A / B.
  struct Loader {
    uint32_t ga[kIA], gb[kIB];
    uint32_t lds0;
    rsrc_t ra, rb;
    int wave;
    template <class AOff, class BOff>
    __device__ __forceinline__ Loader(uint8_t* smem, const uint8_t* A, const uint8_t* B, AOff a_off, BOff b_off) {
      const int lane = threadIdx.x & 63;
      // wave index as a scalar: the LDS addresses of the load instructions are
      // then computed on the scalar unit, with no per-load register round trip
      wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);
      // this lane's source row and chunk for each of the wave's load instructions
      const uint32_t chunk_off = uint32_t((lane & 7) ^ (lane >> 3)) << 4;
#pragma unroll
      for (int i = 0; i < kIA; ++i) ga[i] = a_off((wave * kIA + i) * 8 + (lane >> 3)) + chunk_off;
#pragma unroll
      for (int i = 0; i < kIB; ++i) gb[i] = b_off((wave * kIB + i) * 8 + (lane >> 3)) + chunk_off;
      lds0 = lds_address(smem);
      ra = buffer_rsrc(A);
      rb = buffer_rsrc(B);
    }
    __device__ __forceinline__ void dma_a(int i, uint32_t koff, uint32_t sbase) const {
      lds_dma16(ra, ga[i], koff, sbase + (wave * kIA + i) * 1024);
    }
    __device__ __forceinline__ void dma_b(int i, uint32_t koff, uint32_t sbase) const {
      lds_dma16(rb, gb[i], koff, sbase + kStageA + (wave * kIB + i) * 1024);
    }
    __device__ __forceinline__ void issue(int st, int slot) const {
      const uint32_t koff = uint32_t(st) * kRowBytes, sbase = lds0 + slot * kStage;
#pragma unroll
      for (int i = 0; i < kIA; ++i) dma_a(i, koff, sbase);
#pragma unroll
      for (int i = 0; i < kIB; ++i) dma_b(i, koff, sbase);
    }
  };

  // Issue the copies of K stage `st` (0 or 1) of a tile (nk as in run) into
  // ring slot st: a caller that holds no live data in the ring starts the
  // next tile's copies around the current tile's epilogue.
  template <class AOff, class BOff>
  __device__ __forceinline__ static void issue_stage(uint8_t* smem, const uint8_t* A, const uint8_t* B, AOff a_off,
                                                     BOff b_off, int nk, int st) {
    const Loader ld(smem, A, B, a_off, b_off);
    ld.issue(min(st, (nk >> 1) - 1), st);
  }

  // nk: K / kKPerStage (even).  smem: kSmem bytes.  PRE: stages 0 and 1 were
  // issued by issue_stage, in this order, and stage 1 is the last vector
  // memory load issued (stores may follow it or sit between the two): loads
  // complete in order, so with at most one stage of operations outstanding
  // stage 0 has landed, whatever the stores do.
  template <bool PRE = false, class AOff, class BOff>
  __device__ __forceinline__ static void run(uint8_t* smem, const uint8_t* A, const uint8_t* B, AOff a_off,
                                             BOff b_off, int nk, f32x4 (&acc)[kFM][kFN]) {
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const Loader ld(smem, A, B, a_off, b_off);
    const int wave = ld.wave;
    const int wm = wave / WAVES_N;
    const int wn = wave % WAVES_N;
    const int ns = nk >> 1;   // stages
    auto dma_a = [&](int i, uint32_t koff, uint32_t sbase) { ld.dma_a(i, koff, sbase); };
    auto dma_b = [&](int i, uint32_t koff, uint32_t sbase) { ld.dma_b(i, koff, sbase); };

#pragma unroll
    for (int m = 0; m < kFM; ++m)
#pragma unroll
      for (int n = 0; n < kFN; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int fr = lane & 15;
    const int fc = lane >> 4;
    u32x4 af[2][kFM], bfr[2][kFN];   // fragments of the current and the next sub-step
    // fragments of sub-step h (0 or 1) of the stage in LDS slot `slot`
    auto a_frag = [&](int slot, int h, int m) {
      return *reinterpret_cast<const u32x4*>(smem + slot * kStage + swz(wm * kWTM + m * 16 + fr, 4 * h + fc));
    };
    auto b_frag = [&](int slot, int h, int n) {
      return *reinterpret_cast<const u32x4*>(smem + slot * kStage + kStageA +
                                             swz(wn * kWTN + n * 16 + fr, 4 * h + fc));
    };
    auto mma_one = [&](int r, int i) {
      if constexpr (TRANS)
        Mfma<T>::run(acc[i / kFN][i % kFN], bfr[r][i % kFN], af[r][i / kFN]);
      else
        Mfma<T>::run(acc[i / kFN][i % kFN], af[r][i / kFN], bfr[r][i % kFN]);
    };

    // Every step has the same shape: no branch but the loop's back-edge (a
    // branch inside a step makes the compiler's wait-count analysis wait for
    // the next fragment reads before the current MFMAs).  Past the last stage
    // the loads repeat stage ns - 1 into the slot just released, so that the
    // number of loads in flight, and with it every vmcnt wait, stays uniform;
    // that slot is not read again as a live stage.
    if constexpr (!PRE) {
      ld.issue(0, 0);
      ld.issue(min(1, ns - 1), 1);
    }
    wait_vmcnt<kIA + kIB>();   // stage 0 landed (stage 1 may still be in flight)
    barrier_lds();
#pragma unroll
    for (int m = 0; m < kFM; ++m) af[0][m] = a_frag(0, 0, m);
#pragma unroll
    for (int n = 0; n < kFN; ++n) bfr[0][n] = b_frag(0, 0, n);

    // Sub-step 0 of stage j: MFMAs on the fragments of (j, 0) (register set
    // 0) with the reads of (j, 1) into set 1 spread between them.
    // Sub-step 1: the MFMAs on (j, 1) that need nothing from this step go
    // before the barrier; the barrier needs stage j + 1 landed in every wave
    // and proves every wave has read its last fragments of stage j, so the
    // slot of j takes the load of stage j + 2; after it, each remaining MFMA
    // is followed by one load instruction or one read of (j + 1, 0) into set
    // 0.  Scheduling fences pin this order (left free, the scheduler pairs
    // every fragment read with the MFMA that consumes it).
    constexpr int kMma = kFM * kFN;
    constexpr int kReads = kFM + kFN;
    constexpr int kStride0 = kMma / kReads > 0 ? kMma / kReads : 1;
    constexpr int kComp1 = kIA + kIB + kReads;
    constexpr int kPre1 = kMma > kComp1 ? kMma - kComp1 : 0;
    auto read_into = [&](int r, int slot, int h, int j) {   // j-th fragment read of a sub-step
      if (j < kFM)
        af[r][j] = a_frag(slot, h, j);
      else
        bfr[r][j - kFM] = b_frag(slot, h, j - kFM);
    };
    for (int j = 0; j < ns; ++j) {
      const int cur = j & 1, nxt = cur ^ 1;
      __builtin_amdgcn_sched_barrier(0);
      static_for<0, kMma>([&](auto ii) {
        constexpr int i = decltype(ii)::value;
        mma_one(0, i);
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (i % kStride0 == kStride0 - 1 && i / kStride0 < kReads) {
          read_into(1, cur, 1, i / kStride0);
          __builtin_amdgcn_sched_barrier(0);
        }
      });
      static_for<kMma / kStride0, kReads>([&](auto jj) {   // reads left over when kMma < kReads
        read_into(1, cur, 1, decltype(jj)::value);
        __builtin_amdgcn_sched_barrier(0);
      });
      const uint32_t koff = uint32_t(min(j + 2, ns - 1)) * kRowBytes, sbase = ld.lds0 + cur * kStage;
      if constexpr (EARLY) {
        // slot cur is free once every wave's reads of (j, 1) are done
        barrier_lds();
        __builtin_amdgcn_sched_barrier(0);
        // the copies of stage j + 2, one per MFMA of sub-step 1, then MFMAs up
        // to the point that leaves one MFMA per fragment read of (j + 1, 0)
        constexpr int kL = kIA + kIB;
        constexpr int kB2 = kL > kMma - kReads ? kL : kMma - kReads;
        static_for<0, kB2>([&](auto cc) {
          constexpr int c = decltype(cc)::value;
          if constexpr (c < kMma) {
            mma_one(1, c);
            __builtin_amdgcn_sched_barrier(0);
          }
          if constexpr (c < kIA)
            dma_a(c, koff, sbase);
          else if constexpr (c < kL)
            dma_b(c - kIA, koff, sbase);
          __builtin_amdgcn_sched_barrier(0);
        });
        wait_vmcnt<kL>();   // stage j + 1 landed; stage j + 2 may still be in flight
        barrier_lds();
        __builtin_amdgcn_sched_barrier(0);
        static_for<0, (kMma - kB2 > kReads ? kMma - kB2 : kReads)>([&](auto cc) {
          constexpr int c = decltype(cc)::value;
          if constexpr (kB2 + c < kMma) {
            mma_one(1, kB2 + c);
            __builtin_amdgcn_sched_barrier(0);
          }
          if constexpr (c < kReads) read_into(0, nxt, 0, c);
          __builtin_amdgcn_sched_barrier(0);
        });
        continue;
      }
      static_for<0, kPre1>([&](auto ii) {
        mma_one(1, decltype(ii)::value);
        __builtin_amdgcn_sched_barrier(0);
      });
      wait_vmcnt<0>();
      __syncthreads();
      __builtin_amdgcn_sched_barrier(0);
      static_for<0, (kMma - kPre1 > kComp1 ? kMma - kPre1 : kComp1)>([&](auto cc) {
        constexpr int c = decltype(cc)::value;
        if constexpr (kPre1 + c < kMma) {
          mma_one(1, kPre1 + c);
          __builtin_amdgcn_sched_barrier(0);
        }
        if constexpr (c < kIA)
          dma_a(c, koff, sbase);
        else if constexpr (c < kIA + kIB)
          dma_b(c - kIA, koff, sbase);
        else if constexpr (c < kComp1)
          read_into(0, nxt, 0, c - kIA - kIB);
        __builtin_amdgcn_sched_barrier(0);
      });
    }
    wait_vmcnt<0>();
    __syncthreads();   // the caller may reuse the LDS
  }
};

// 256 x 256 tile with the waves of TileMma<T, 256, 256, 4, 2> (64 x 128 each,
// same accumulator layout) run as two groups that take turns on the matrix
// cores.  Waves 0-3 (group 0: rows 0-127 of the tile) and waves 4-7 (group 1:
// rows 128-255) put one wave of each group on every SIMD.  Each K sub-step
// (64 bytes of K) is one phase per group: a load phase (the sub-step's 12
// fragment reads, copies into the ring, waits) and an MFMA phase (32 MFMAs
// on registers).  Group 1 runs one phase behind group 0, and a workgroup
// barrier ends every phase, so that on each SIMD one wave issues MFMAs back
// to back while the other loads: the LDS reads of one group overlap the
// other's MFMAs instead of all waves reading at once after a barrier.
//
// Ring of two stage slots, as in TileMma.  Copies of stage s + 2 go into the
// slot of stage s as soon as no wave reads that part any more, split so that
// every copy has about four phases to land:
//   A rows 0-127 (read by group 0 only): group 1, in its load phase of
//     sub-step (s, 1), after group 0's last read of them;
//   A rows 128-255: group 0, in its load phase of (s + 1, 0);
//   B: group 1, in its load phase of (s + 1, 0).
// A group waits for its copies of a stage at the end of the load phase just
// before the first read of that stage by any wave, so the barrier that ends
// the phase publishes them.  Past the last stage the copies repeat stage
// ns - 1 (same data, into parts no wave reads any more), keeping every wait
// count uniform.
template <typename T, bool TRANS = false>
struct PingPongMma {
  using Base = TileMma<T, 256, 256, 4, 2, TRANS>;
  static constexpr int kWaves = 8, kThreads = 512;
  static constexpr int kWTM = Base::kWTM, kWTN = Base::kWTN, kFM = Base::kFM, kFN = Base::kFN;
  static constexpr int kRowBytes = Base::kRowBytes, kStageA = Base::kStageA, kStage = Base::kStage;
  static constexpr int kSmem = Base::kSmem;
  static constexpr int kKPerStage = Base::kKPerStage;
  static constexpr int kIH = 4;   // copy instructions per wave for half of A (128 rows / 8 / 4 waves)
  static constexpr int kIB = 8;   // for B (256 rows / 8 / 4 waves)
  static_assert(kFM == 4 && kFN == 8, "ping-pong layout");

  __device__ __forceinline__ static int swz(int r, int c) { return Base::swz(r, c); }

  // the wave's copies: group 0 copies A rows 128-255, group 1 A rows 0-127 and B
  struct Loader {
    uint32_t ga[kIH], gb[kIB];
    uint32_t lds0;
    rsrc_t ra, rb;
    int q, grp;   // index within the group, group
    template <class AOff, class BOff>
    __device__ __forceinline__ Loader(uint8_t* smem, const uint8_t* A, const uint8_t* B, AOff a_off, BOff b_off) {
      const int lane = threadIdx.x & 63;
      const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);
      q = wave & 3;
      grp = wave >> 2;
      const uint32_t chunk_off = uint32_t((lane & 7) ^ (lane >> 3)) << 4;
      const int a_first = grp ? 0 : 128;
#pragma unroll
      for (int i = 0; i < kIH; ++i) ga[i] = a_off(a_first + (q * kIH + i) * 8 + (lane >> 3)) + chunk_off;
#pragma unroll
      for (int i = 0; i < kIB; ++i) gb[i] = b_off((q * kIB + i) * 8 + (lane >> 3)) + chunk_off;
      lds0 = lds_address(smem);
      ra = buffer_rsrc(A);
      rb = buffer_rsrc(B);
    }
    // this wave's half of A of stage st into ring slot `slot`
    __device__ __forceinline__ void copy_a(int st, int slot) const {
      const uint32_t koff = uint32_t(st) * kRowBytes;
      const uint32_t base = lds0 + slot * kStage + ((grp ? 0 : 16) + q * kIH) * 1024;
#pragma unroll
      for (int i = 0; i < kIH; ++i) lds_dma16(ra, ga[i], koff, base + i * 1024);
    }
    // this wave's share of B of stage st (group 1 only)
    __device__ __forceinline__ void copy_b(int st, int slot) const {
      const uint32_t koff = uint32_t(st) * kRowBytes;
      const uint32_t base = lds0 + slot * kStage + kStageA + q * kIB * 1024;
#pragma unroll
      for (int i = 0; i < kIB; ++i) lds_dma16(rb, gb[i], koff, base + i * 1024);
    }
  };

  // Copies of stage `st` (0 or 1) of a tile into ring slot st, as run expects
  // them when PRE: stage 0 whole (every wave its TileMma share), stage 1 split
  // by group (group 0: A rows 128-255; group 1: A rows 0-127, then B).
  template <class AOff, class BOff>
  __device__ __forceinline__ static void issue_stage(uint8_t* smem, const uint8_t* A, const uint8_t* B, AOff a_off,
                                                     BOff b_off, int nk, int st) {
    if (st == 0) {
      Base::issue_stage(smem, A, B, a_off, b_off, nk, 0);
    } else {
      const Loader ld(smem, A, B, a_off, b_off);
      const int s1 = min(1, (nk >> 1) - 1);
      ld.copy_a(s1, 1);
      if (ld.grp) ld.copy_b(s1, 1);
    }
  }

  template <bool PRE = false, class AOff, class BOff>
  __device__ __forceinline__ static void run(uint8_t* smem, const uint8_t* A, const uint8_t* B, AOff a_off,
                                             BOff b_off, int nk, f32x4 (&acc)[kFM][kFN]) {
    if constexpr (!PRE) {
      issue_stage(smem, A, B, a_off, b_off, nk, 0);
      issue_stage(smem, A, B, a_off, b_off, nk, 1);
    }
    const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);
    if (wave >= 4)
      group_loop<1>(smem, A, B, a_off, b_off, nk, acc);
    else
      group_loop<0>(smem, A, B, a_off, b_off, nk, acc);
    wait_vmcnt<0>();
    __syncthreads();   // the caller may reuse the LDS
  }

 private:
  template <int G, class AOff, class BOff>
  __device__ __forceinline__ static void group_loop(uint8_t* smem, const uint8_t* A, const uint8_t* B, AOff a_off,
                                                    BOff b_off, int nk, f32x4 (&acc)[kFM][kFN]) {
    const int lane = threadIdx.x & 63;
    const Loader ld(smem, A, B, a_off, b_off);
    const int wave = int(threadIdx.x) >> 6;
    const int wm = wave / 2, wn = wave % 2;
    const int ns = nk >> 1;
    const int fr = lane & 15, fc = lane >> 4;

#pragma unroll
    for (int m = 0; m < kFM; ++m)
#pragma unroll
      for (int n = 0; n < kFN; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};

    u32x4 af[2][kFM], bfr[2][kFN];
    auto reads = [&](int r, int slot, int h) {
      const uint8_t* st = smem + slot * kStage;
#pragma unroll
      for (int m = 0; m < kFM; ++m)
        af[r][m] = *reinterpret_cast<const u32x4*>(st + swz(wm * kWTM + m * 16 + fr, 4 * h + fc));
#pragma unroll
      for (int n = 0; n < kFN; ++n)
        bfr[r][n] = *reinterpret_cast<const u32x4*>(st + kStageA + swz(wn * kWTN + n * 16 + fr, 4 * h + fc));
    };
    auto mfmas = [&](int r) {
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < kFM * kFN; ++i) {
        if constexpr (TRANS)
          Mfma<T>::run(acc[i / kFN][i % kFN], bfr[r][i % kFN], af[r][i / kFN]);
        else
          Mfma<T>::run(acc[i / kFN][i % kFN], af[r][i / kFN], bfr[r][i % kFN]);
      }
      __builtin_amdgcn_sched_barrier(0);
    };
    auto phase_end = [&]() {
      __builtin_amdgcn_sched_barrier(0);
      barrier_lds();
      __builtin_amdgcn_sched_barrier(0);
    };

    // stage 0 landed in every wave (stage 1 may be in flight), then published
    if constexpr (G == 0)
      wait_vmcnt<kIH>();
    else
      wait_vmcnt<kIH + kIB>();
    phase_end();
    if constexpr (G == 1) phase_end();   // one phase behind group 0

    for (int s = 0; s < ns; ++s) {
      const int slot = s & 1;
      // load phase of sub-step (s, 0)
      reads(0, slot, 0);
      if (s > 0) {
        const int st = min(s + 1, ns - 1);
        if constexpr (G == 0)
          ld.copy_a(st, slot ^ 1);
        else
          ld.copy_b(st, slot ^ 1);
      }
      if constexpr (G == 0) wait_vmcnt<kIH>();   // A rows 128-255 of stage s landed (stage s + 1's in flight)
      phase_end();
      mfmas(0);
      phase_end();
      // load phase of sub-step (s, 1)
      reads(1, slot, 1);
      if constexpr (G == 1) {
        wait_lgkmcnt0();
        ld.copy_a(min(s + 2, ns - 1), slot);
        wait_vmcnt<kIH>();   // A rows 0-127 and B of stage s + 1 landed
      }
      phase_end();
      mfmas(1);
      phase_end();
    }
    if constexpr (G == 0) phase_end();   // matches group 1's extra phase
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
