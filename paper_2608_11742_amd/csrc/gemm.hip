// Projection GEMMs of the transformer layer with fused epilogues:
//   resid  : x += a W^T                      (O and down projections)
//   swiglu : f = silu(a Wg^T) * (a Wu^T)     (gate/up projection)
//   qkv    : q, k, v = a Wqkv^T, rotary embedding on q and k, scattered to
//            head-major Q/K and transposed V
// 256x256 output tiles, 8 waves of 64x128, bf16 (or fp32) MFMA, fp32 accumulate;
// fewer rows take the smaller tile configurations below.
//
// Few rows (a 512-row forward has 32 output tiles in the O and down
// projections for 256 CUs): the K range is split into parts, every part
// writes an fp32 partial tile to the workspace, and a reduction kernel adds
// the parts in a fixed order (deterministic) and applies the epilogue.
#include <algorithm>

#include "kernels.h"
#include "mainloop.h"

namespace dllm {

namespace {

// Tile configurations; Big and Small with waves of 64 x 128 (the epilogues' layout):
// Big 256 x 256 with 8 waves (two per SIMD, one workgroup per CU); Small
// 64 x 256 with 2 waves for GEMMs of at most kSmallM rows, where a 256-row
// tile would mostly multiply clamped duplicate rows (two workgroups per CU).
// EARLY: the TileMma schedule that hands a consumed ring slot to its next
// copies half a stage sooner (measured faster where the weights stream from
// HBM at one tile per CU: 4-10% on the Quad and Mid launches, no change on
// Small).
template <int BM_, int BN_, int WM_, int WN_, int MIN_BLOCKS, bool EARLY = false>
struct GemmCfg {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, kThreads = WM_ * WN_ * 64, kMinBlocks = MIN_BLOCKS;
  static constexpr bool kEarly = EARLY;
};
using Big = GemmCfg<256, 256, 4, 2, 2>;
using Small = GemmCfg<64, 256, 1, 2, 2>;
// few rows (a block forward over a cached prefix, the suffix of a decode):
// 128 x 256 tiles of 8 waves of 32 x 128 (two per SIMD, as Big), so that a
// 65-256-row projection wastes fewer clamped rows and needs half the split-K
// parts of 256-row tiles
using Quad = GemmCfg<128, 256, 4, 2, 1, true>;
// gate/up with 257-512 rows: 256 x 192 tiles (waves of 64 x 96, 48 gate + 48
// up rows each) give 2 x F / 96 = 256 workgroups for the 8B shape, one per CU,
// where 256 x 256 tiles leave a quarter of the CUs idle; also the split-K
// parts of the QKV projection over 129-512 rows (qkv_mid_parts)
using Mid = GemmCfg<256, 192, 4, 2, 2, true>;
constexpr int kBN = 256;          // Big and Small: column tile of the split-K partials and the QKV / residual launches
constexpr int kGroupM = 8;
#ifndef DLLM_PINGPONG
#define DLLM_PINGPONG 1
#endif
constexpr bool kPingPong = DLLM_PINGPONG;

// mainloop of a tile configuration: bf16 256 x 256 tiles take the two-group
// schedule (PingPongMma), every other configuration TileMma
template <typename T, class Cfg, bool TRANS>
using MainLoop =
    std::conditional_t<kPingPong && std::is_same_v<T, bf16_t> && Cfg::BM == 256 && Cfg::BN == 256 && Cfg::WM == 4 &&
                           Cfg::WN == 2,
                       PingPongMma<T, TRANS>, TileMma<T, Cfg::BM, Cfg::BN, Cfg::WM, Cfg::WN, TRANS, Cfg::kEarly>>;
#ifndef DLLM_SMALL_M_MAX
#define DLLM_SMALL_M_MAX 64
#endif
constexpr int kSmallM = DLLM_SMALL_M_MAX;

// Row tile of a projection of M rows: Small up to kSmallM rows; Quad where it
// measured faster than Big (the d-wide O projection up to 512 rows, the
// F-deep down projection at 1, 2 or 4 row tiles up to 512 rows, QKV and
// gate/up up to 128); Big above.
int tile_rows(int kind, int M, int N, int K) {
  if (M <= kSmallM) return Small::BM;
  if (kind == GEMM_KIND_RESID && K > N && M <= 512) {
    // the F-deep down projection: 128-row tiles when their split-K parts fill
    // the CUs exactly (1, 2 or 4 row tiles), else 256-row tiles
    const int tm = cdiv(M, Quad::BM);
    return (tm & (tm - 1)) == 0 ? Quad::BM : Big::BM;
  }
  const int quad_max = kind == GEMM_KIND_RESID ? 512 : 128;
  return M <= quad_max ? Quad::BM : Big::BM;
}

// Split-K parts of the QKV projection over 129-512 rows take 256 x 192 tiles:
// 3 d / 192 column tiles by 1 or 2 row tiles, times the parts, fill the 256
// CUs exactly for the 8B shape (128 x 2 or 64 x 4), where 256 x 256 tiles
// leave a quarter of them idle (96 x 2 or 48 x 4)
static bool qkv_mid_parts(int M, int N) { return M > 128 && M <= 512 && N % Mid::BN == 0; }

// EPI_PART / EPI_PART_GU: split-K partial tiles (GU: the gate/up row pairing
// of EPI_SWIGLU) written to part[split][M][np]
enum { EPI_RESID = 0, EPI_SWIGLU = 1, EPI_QKV = 2, EPI_PART = 3, EPI_PART_GU = 4 };

struct EpiParams {
  float* x;          // resid: fp32 residual
  int ldx;
  void* out;         // swiglu: [M][F]
  int F;
  QkvOut qkv;
  float* part;       // split-K partials [splits][M][np]
  int np;
};

// gate/up epilogue of one tile: out = silu(gate) * up.  The blocks are
// transposed (TileMma TRANS): lane l holds row 16 m + l % 16, columns
// 16 n + 4 (l / 16) + i of the wave tile; gate block n pairs with up block
// n + kFN / 2, so each lane stores 4 consecutive outputs at once.
template <typename T, class Cfg, class TM>
__device__ __forceinline__ void swiglu_store(const f32x4 (&acc)[TM::kFM][TM::kFN], int m0, int tn, int M,
                                             const EpiParams& ep) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / Cfg::WN, wn = wave % Cfg::WN;
  T* out = reinterpret_cast<T*>(ep.out);
  constexpr int kOC = TM::kWTN / 2, kNG = TM::kFN / 2;
  const int jw = tn * (Cfg::BN / 2) + wn * kOC, rw = m0 + wm * TM::kWTM;   // wave tile origin
  const int j0 = jw + 4 * (lane >> 4), r0 = rw + (lane & 15);
  // all values first (independent chains the scheduler can interleave),
  // then the stores: unguarded when the whole wave tile is in range
  float v[TM::kFM][kNG][4];
#pragma unroll
  for (int m = 0; m < TM::kFM; ++m)
#pragma unroll
    for (int n = 0; n < kNG; ++n)
#pragma unroll
      for (int i = 0; i < 4; ++i) v[m][n][i] = silu_fast(acc[m][n][i]) * acc[m][n + kNG][i];
  const bool vec = (ep.F % 4) == 0 && (reinterpret_cast<uintptr_t>(out) & (4 * sizeof(T) - 1)) == 0;
  if (vec && rw + TM::kWTM <= M && jw + kOC <= ep.F) {
#pragma unroll
    for (int m = 0; m < TM::kFM; ++m)
#pragma unroll
      for (int n = 0; n < kNG; ++n) {
        T* dst = out + size_t(r0 + 16 * m) * ep.F + j0 + 16 * n;
        if constexpr (Elem<T>::bytes == 2)
          *reinterpret_cast<u32x2*>(dst) =
              u32x2{pack_bf16x2(v[m][n][0], v[m][n][1]), pack_bf16x2(v[m][n][2], v[m][n][3])};
        else
          *reinterpret_cast<f32x4*>(dst) = f32x4{v[m][n][0], v[m][n][1], v[m][n][2], v[m][n][3]};
      }
  } else {
#pragma unroll
    for (int m = 0; m < TM::kFM; ++m)
#pragma unroll
      for (int n = 0; n < kNG; ++n)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = r0 + 16 * m, j = j0 + 16 * n + i;
          if (row < M && j < ep.F) store_f(out + size_t(row) * ep.F + j, v[m][n][i]);
        }
  }
}

// B row of local tile row r in a gate/up tile: each wave column of kWTN rows
// pairs kWTN / 2 gate rows with the kWTN / 2 up rows of the same outputs
template <class Cfg, class TM>
__device__ __forceinline__ int gu_row(int r, int tn, int F) {
  constexpr int kHalf = TM::kWTN / 2;
  const int wn = r / TM::kWTN, rr = r % TM::kWTN;
  const int j = min(tn * (Cfg::BN / 2) + wn * kHalf + rr % kHalf, F - 1);
  return rr < kHalf ? j : F + j;
}

// in-sequence position id of row `row` of the QKV projection (absolute, packed-lookahead aware)
__device__ __forceinline__ int qkv_pos(const QkvOut& o, int row) {
  const int r = row % o.seq;
  return o.pos_offset + (o.pack_B && r >= o.pack_S ? o.pack_b0 + ((r - o.pack_S) & (o.pack_B - 1)) : r);
}

// Tile and K part of a split-K workgroup (grid: tiles x parts).  Workgroups
// are dispatched to the 8 XCDs round-robin by linear id; when the part count
// divides 8 or is a multiple of 8, each XCD gets whole parts (or an even share
// of one part's tiles, the row tiles of a column tile together), so that all
// readers of an A or B panel of a part share one L2 and the panel is fetched
// once, instead of once per XCD.  The part a workgroup computes, and so the
// summation order, does not depend on this mapping.
__device__ __forceinline__ void map_split_tile(int tiles_m, int tiles_n, int parts, int& tm, int& tn, int& part) {
  const int T = tiles_m * tiles_n;
  const int L = int(blockIdx.x) + int(gridDim.x) * int(blockIdx.y);
  const int xcd = L % 8, local = L / 8;
  int j;
  if (parts % 8 == 0) {
    part = xcd * (parts / 8) + local / T;
    j = local % T;
  } else if (8 % parts == 0 && T % (8 / parts) == 0) {
    const int per = 8 / parts;   // XCDs per part
    part = xcd / per;
    j = (xcd % per) * (T / per) + local;
  } else {
    part = blockIdx.y;
    map_tile(blockIdx.x, gridDim.x, tiles_m, tiles_n, kGroupM, tm, tn);
    return;
  }
  tm = j % tiles_m;
  tn = j / tiles_m;
}

// HD: head_dim of the QKV epilogue (compile-time, so the rotary partner block
// index stays static and the accumulators stay in registers); 0 otherwise.
template <typename T, int EPI, int HD, class Cfg>
__global__ __launch_bounds__(Cfg::kThreads, Cfg::kMinBlocks) void gemm_kernel(const T* __restrict__ A, int lda,
                                                                const T* __restrict__ B, int ldb, int M, int N,
                                                                int K, int tiles_m, int tiles_n, EpiParams ep) {
  constexpr int kBM = Cfg::BM, kWavesN = Cfg::WN;
  constexpr bool kTrans = EPI == EPI_SWIGLU;
  using TM = MainLoop<T, Cfg, kTrans>;
  constexpr bool kSplit = EPI == EPI_PART || EPI == EPI_PART_GU;
  __shared__ __attribute__((aligned(16))) uint8_t smem[TM::kSmem];
  int tm, tn, part = 0;
  if constexpr (kSplit)
    map_split_tile(tiles_m, tiles_n, gridDim.y, tm, tn, part);
  else
    map_tile(blockIdx.x, gridDim.x, tiles_m, tiles_n, kGroupM, tm, tn);
  const int m0 = tm * kBM;
  const uint32_t a_row_bytes = uint32_t(lda) * sizeof(T);
  const uint32_t b_row_bytes = uint32_t(ldb) * sizeof(T);
  // K stages of this part (128 bytes of every row per stage)
  int st0 = 0, nst = K / (2 * TM::kKPerStage);
  if constexpr (kSplit) {
    const int all = nst;
    st0 = part * all / int(gridDim.y);
    nst = (part + 1) * all / int(gridDim.y) - st0;
  }
  const uint32_t k_bytes = uint32_t(st0) * TM::kRowBytes;
  auto a_off = [&](int r) -> uint32_t { return uint32_t(min(m0 + r, M - 1)) * a_row_bytes + k_bytes; };
  auto b_off = [&](int r) -> uint32_t {
    int row;
    if constexpr (EPI == EPI_SWIGLU || EPI == EPI_PART_GU) {
      row = gu_row<Cfg, TM>(r, tn, ep.F);   // BN rows -> BN / 2 outputs
    } else {
      row = min(tn * Cfg::BN + r, N - 1);
    }
    return uint32_t(row) * b_row_bytes + k_bytes;
  };
  f32x4 acc[TM::kFM][TM::kFN];
  TM::run(smem, reinterpret_cast<const uint8_t*>(A), reinterpret_cast<const uint8_t*>(B), a_off, b_off, 2 * nst,
          acc);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / kWavesN, wn = wave % kWavesN;
  const int row_base = m0 + wm * TM::kWTM + 4 * (lane >> 4);
  const int lc = lane & 15;

  if constexpr (kSplit) {
    // the fp32 partial tile through LDS as in the residual epilogue, 16-byte
    // stores along rows of part[split]: each wave stages RG rows by up to 64
    // columns of its tile at a time (a 96-column wave tile as 64 + 32); RG is
    // halved where the staging of all waves would not fit in the ring
    static_assert((TM::kWTM % 64 == 0 || TM::kWTM == 32) &&
                      (TM::kWTN == 128 || (TM::kWTN == 96 && EPI == EPI_PART)),
                  "partial epilogue tiling");
    constexpr int RG0 = TM::kWTM >= 64 ? 64 : TM::kWTM;
    constexpr int RG = TM::kWaves * RG0 * 64 * 4 <= TM::kSmem ? RG0 : RG0 / 2;   // rows per staged group
    static_assert(TM::kWaves * RG * 64 * 4 <= TM::kSmem, "staging inside the ring");
    uint8_t* st = smem + wave * (RG * 64 * 4);
    auto slot_of = [](int r, int c4) { return r * 256 + (((c4 ^ (r & 15))) << 4); };
    float* P = ep.part + size_t(part) * M * ep.np;
#pragma unroll
    for (int g = 0; g < TM::kWTM / RG; ++g) {   // row groups of the wave tile
      const int r0 = m0 + wm * TM::kWTM + RG * g;
      static_for<0, cdiv(TM::kFN, 4)>([&](auto hh) {   // column groups of up to 64
        constexpr int h = decltype(hh)::value;
        constexpr int NB = TM::kFN - 4 * h < 4 ? TM::kFN - 4 * h : 4;   // 16-column blocks of the group
        constexpr int CH = 4 * NB;                                      // 16-byte chunks of a staged row
#pragma unroll
        for (int m = 0; m < RG / 16; ++m)
#pragma unroll
          for (int nn = 0; nn < NB; ++nn)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int r = m * 16 + 4 * (lane >> 4) + i, c = nn * 16 + lc;
              *reinterpret_cast<float*>(st + slot_of(r, c >> 2) + (c & 3) * 4) = acc[(RG / 16) * g + m][4 * h + nn][i];
            }
        const int c0 = tn * Cfg::BN + wn * TM::kWTN + 64 * h;
#pragma unroll
        for (int j = 0; j < RG * CH / 64; ++j) {
          const int q = lane + 64 * j, r = q / CH, c4 = q % CH;
          const int row = r0 + r;
          if (row < M)
            *reinterpret_cast<f32x4*>(P + size_t(row) * ep.np + c0 + 4 * c4) =
                *reinterpret_cast<const f32x4*>(st + slot_of(r, c4));
        }
      });
    }
  } else if constexpr (EPI == EPI_RESID) {
    // x += acc through LDS: each wave stages half of its 64 x 128 tile at a
    // time (64 x 64 fp32, 16 KB, in its own region of the idle ring), rows of
    // 16 chunks of 4 floats with chunk c of row r in slot c ^ (r % 16), so
    // both the MFMA-layout writes and the row reads are conflict-free; then
    // every lane reads 16 bytes of x per access, all loads first (clamped
    // into the matrix) and the guarded stores after them.
    static_assert((TM::kWTM % 64 == 0 || TM::kWTM == 32) && TM::kWTN == 128, "resid epilogue tiling");
    constexpr int RG = TM::kWTM >= 64 ? 64 : TM::kWTM;   // rows per staged group
    static_assert(TM::kWaves * RG * 64 * 4 <= TM::kSmem, "staging inside the ring");
    uint8_t* st = smem + wave * (RG * 64 * 4);
    auto slot_of = [](int r, int c4) { return r * 256 + (((c4 ^ (r & 15))) << 4); };
#pragma unroll
    for (int g = 0; g < TM::kWTM / RG; ++g) {   // row groups of the wave tile
      const int r0 = m0 + wm * TM::kWTM + RG * g;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int m = 0; m < RG / 16; ++m)
#pragma unroll
          for (int nn = 0; nn < 4; ++nn)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int r = m * 16 + 4 * (lane >> 4) + i, c = nn * 16 + lc;
              *reinterpret_cast<float*>(st + slot_of(r, c >> 2) + (c & 3) * 4) = acc[(RG / 16) * g + m][4 * h + nn][i];
            }
        const int c0 = tn * Cfg::BN + wn * TM::kWTN + 64 * h;
        f32x4 xv[RG / 4];
#pragma unroll
        for (int j = 0; j < RG / 4; ++j) {
          const int q = lane + 64 * j, r = q >> 4, c4 = q & 15;
          const int row = min(r0 + r, M - 1), col = min(c0 + 4 * c4, N - 4);
          xv[j] = *reinterpret_cast<const f32x4*>(ep.x + size_t(row) * ep.ldx + col);
        }
#pragma unroll
        for (int j = 0; j < RG / 4; ++j) {
          const int q = lane + 64 * j, r = q >> 4, c4 = q & 15;
          const int row = r0 + r, col = c0 + 4 * c4;
          const f32x4 a = *reinterpret_cast<const f32x4*>(st + slot_of(r, c4));
          if (row < M && col < N) *reinterpret_cast<f32x4*>(ep.x + size_t(row) * ep.ldx + col) = xv[j] + a;
        }
      }
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    swiglu_store<T, Cfg, TM>(acc, m0, tn, M, ep);
  } else {  // EPI_QKV
    static_assert(HD == 64 || HD == 128, "head_dim");
    const QkvOut& o = ep.qkv;
    constexpr int hd = HD, half = HD / 2, pair = HD / 32;  // partner block distance
    const int wcol0 = tn * Cfg::BN + wn * TM::kWTN;        // first column of this wave tile
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
      const int r0 = m0 + wm * TM::kWTM;
      if (which < 2) {
        // Q, K: stage the wave's 64 x 128 bf16 tile in its own region of the
        // idle ring (rows of 16 chunks; chunk c of row r in slot
        // c ^ 2 ((r / 4) % 4), so the 4 row groups of a store hit different
        // banks), then write 16-byte chunks along head_dim.  The wave reads
        // back only what it wrote: its LDS operations complete in order, so
        // no barrier.
        static_assert(TM::kWTN == 128, "qkv staging: 16 chunks per row");
        static_assert(TM::kWaves * TM::kWTM * TM::kWTN * 2 <= TM::kSmem, "qkv staging inside the ring");
        uint8_t* st = smem + wave * (TM::kWTM * TM::kWTN * 2);
        auto off = [](int r, int c16) { return r * 256 + ((c16 ^ (((r >> 2) & 3) << 1)) << 4); };
#pragma unroll
        for (int m = 0; m < TM::kFM; ++m)
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int n = 0; n < TM::kFN; ++n) {
              const int r = m * 16 + 4 * (lane >> 4) + i, c = n * 16 + lc;
              *reinterpret_cast<uint16_t*>(st + off(r, c >> 3) + (c & 7) * 2) = uint16_t(pack_bf16x2(acc[m][n][i], 0.f));
            }
        uint16_t* dst = reinterpret_cast<uint16_t*>(which == 0 ? o.q : o.k);
#pragma unroll
        for (int it = 0; it < TM::kWTM * TM::kWTN / 8 / 64; ++it) {
          const int q = lane + 64 * it, r = q / 16, c16 = q % 16;
          const int row = r0 + r;
          if (row >= M) continue;
          const int b = row / o.seq, sp = row % o.seq;
          const int cin = cin0 + c16 * 8, h = cin / hd, dim = cin % hd;
          *reinterpret_cast<u32x4*>(dst + (size_t(b * o.H + h) * o.seq + sp) * hd + dim) =
              *reinterpret_cast<const u32x4*>(st + off(r, c16));
        }
      } else {
        // V^T in IEEE binary16 (see pack_vt2).  A lane's 4 values of a block
        // are 4 consecutive positions of one head dim (8 contiguous bytes of
        // a V^T row).  A 64-row wave tile inside one sequence is staged
        // transposed in the wave's own region of the idle ring, [dim][64
        // positions] in rows of 8 chunks of 8 positions (chunk c of dim row d
        // in slot c ^ (d % 8)), and written back with 16 bytes per lane, 8
        // lanes per whole 128-byte V^T row; other tiles store the 8-byte
        // pieces straight from registers.
        bool staged = false;
        if constexpr (TM::kWTM == 64) {
          static_assert(TM::kWaves * 64 * 128 * 2 <= TM::kSmem, "v staging inside the ring");
          if (o.seq % 64 == 0 && r0 + 64 <= M && o.vt_ld % 8 == 0) {
            uint8_t* st = smem + wave * (64 * 128 * 2);
            auto voff = [](int d, int p) { return d * 128 + (((p >> 3) ^ (d & 7)) << 4) + (p & 7) * 2; };
#pragma unroll
            for (int m = 0; m < TM::kFM; ++m)
#pragma unroll
              for (int n = 0; n < TM::kFN; ++n)
                *reinterpret_cast<u32x2*>(st + voff(n * 16 + lc, m * 16 + 4 * (lane >> 4))) =
                    u32x2{pack_vt2(acc[m][n][0], acc[m][n][1]), pack_vt2(acc[m][n][2], acc[m][n][3])};
            const int b = r0 / o.seq, sp0 = r0 - b * o.seq;
            uint16_t* vt = reinterpret_cast<uint16_t*>(o.vt);
#pragma unroll
            for (int it = 0; it < 128 * 8 / 64; ++it) {
              const int q = lane + 64 * it, d = q >> 3, c = q & 7;
              const int cin = cin0 + d, h = cin / hd, dim = cin % hd;
              *reinterpret_cast<u32x4*>(vt + (size_t(b * o.H + h) * hd + dim) * o.vt_ld + sp0 + c * 8) =
                  *reinterpret_cast<const u32x4*>(st + d * 128 + ((c ^ (d & 7)) << 4));
            }
            staged = true;
          }
        }
        if (!staged) {
          uint16_t* vt = reinterpret_cast<uint16_t*>(o.vt);
          const bool vec4 = (o.seq % 4) == 0 && (o.vt_ld % 4) == 0;
#pragma unroll
          for (int m = 0; m < TM::kFM; ++m) {
            const int row = row_base + m * 16;   // rows row .. row + 3
            if (row >= M) continue;
            const int b = row / o.seq, sp = row - b * o.seq;
#pragma unroll
            for (int n = 0; n < TM::kFN; ++n) {
              const int cin = cin0 + n * 16 + lc, h = cin / hd, dim = cin % hd;
              if (vec4 && row + 3 < M) {
                *reinterpret_cast<u32x2*>(vt + (size_t(b * o.H + h) * hd + dim) * o.vt_ld + sp) =
                    u32x2{pack_vt2(acc[m][n][0], acc[m][n][1]), pack_vt2(acc[m][n][2], acc[m][n][3])};
              } else {
                for (int i = 0; i < 4 && row + i < M; ++i) {
                  const int bi = (row + i) / o.seq, si = (row + i) - bi * o.seq;
                  vt[(size_t(bi * o.H + h) * hd + dim) * o.vt_ld + si] = uint16_t(pack_vt2(acc[m][n][i], 0.f));
                }
              }
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

// Gate/up + SwiGLU over all tiles with one workgroup per CU, each taking
// tiles blockIdx.x, blockIdx.x + gridDim.x, ...: the copies of a tile's first
// K stage are issued before the previous tile's epilogue (which keeps its
// data in registers) and those of the second after its stores, so the first
// stage's latency hides behind the epilogue and the first wait does not
// wait for the stores.
template <typename T, class Cfg>
__global__ __launch_bounds__(Cfg::kThreads, Cfg::kMinBlocks) void gemm_swiglu_persist_kernel(
    const T* __restrict__ A, int lda, const T* __restrict__ B, int M, int K, int tiles_m, int tiles_n, EpiParams ep) {
  using TM = MainLoop<T, Cfg, true>;
  __shared__ __attribute__((aligned(16))) uint8_t smem[TM::kSmem];
  const int ntiles = tiles_m * tiles_n;
  const int nk = K / TM::kKPerStage;
  const uint8_t* A8 = reinterpret_cast<const uint8_t*>(A);
  const uint8_t* B8 = reinterpret_cast<const uint8_t*>(B);
  const uint32_t a_row_bytes = uint32_t(lda) * sizeof(T), b_row_bytes = uint32_t(K) * sizeof(T);
  auto a_off_of = [=](int m0) { return [=](int r) -> uint32_t { return uint32_t(min(m0 + r, M - 1)) * a_row_bytes; }; };
  auto b_off_of = [=](int tn) {
    return [=](int r) -> uint32_t { return uint32_t(gu_row<Cfg, TM>(r, tn, ep.F)) * b_row_bytes; };
  };
  int id = blockIdx.x, tm, tn;
  map_tile(id, ntiles, tiles_m, tiles_n, kGroupM, tm, tn);
  TM::issue_stage(smem, A8, B8, a_off_of(tm * Cfg::BM), b_off_of(tn), nk, 0);
  TM::issue_stage(smem, A8, B8, a_off_of(tm * Cfg::BM), b_off_of(tn), nk, 1);
  for (;;) {
    f32x4 acc[TM::kFM][TM::kFN];
    TM::template run<true>(smem, A8, B8, a_off_of(tm * Cfg::BM), b_off_of(tn), nk, acc);
    const int next = id + int(gridDim.x);
    int tm1 = 0, tn1 = 0;
    if (next < ntiles) {
      map_tile(next, ntiles, tiles_m, tiles_n, kGroupM, tm1, tn1);
      TM::issue_stage(smem, A8, B8, a_off_of(tm1 * Cfg::BM), b_off_of(tn1), nk, 0);
    }
    swiglu_store<T, Cfg, TM>(acc, tm * Cfg::BM, tn, M, ep);
    if (next >= ntiles) break;
    TM::issue_stage(smem, A8, B8, a_off_of(tm1 * Cfg::BM), b_off_of(tn1), nk, 1);
    id = next;
    tm = tm1;
    tn = tn1;
  }
}

// compute units of the current device (cached per device)
int device_cus() {
  static int cus[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cus[dev] = n;
  }
  return cus[dev];
}

template <typename T, int EPI, int HD, class Cfg>
hipError_t launch_cfg(const void* A, int lda, const void* B, int ldb, int M, int N, int K, int tiles_n,
                      const EpiParams& ep, hipStream_t s, int splits) {
  // the mainloop runs stages in pairs
  constexpr int kStageK = 2 * TileMma<T, Cfg::BM, Cfg::BN, Cfg::WM, Cfg::WN>::kKPerStage;
  if (K <= 0 || K % kStageK || splits < 1 || splits > K / kStageK) return hipErrorInvalidValue;
  const int tiles_m = cdiv(M, Cfg::BM);
  const int grid = tiles_m * tiles_n;
  hipLaunchKernelGGL((gemm_kernel<T, EPI, HD, Cfg>), dim3(grid, splits), dim3(Cfg::kThreads), 0, s,
                     static_cast<const T*>(A), lda, static_cast<const T*>(B), ldb, M, N, K, tiles_m, tiles_n, ep);
  return hipGetLastError();
}

// bm: the row tile (tile_rows)
template <typename T, int EPI, int HD = 0>
hipError_t launch(int bm, const void* A, int lda, const void* B, int ldb, int M, int N, int K, int tiles_n,
                  const EpiParams& ep, hipStream_t s, int splits = 1) {
  if (bm == Small::BM) return launch_cfg<T, EPI, HD, Small>(A, lda, B, ldb, M, N, K, tiles_n, ep, s, splits);
  if (bm == Quad::BM) return launch_cfg<T, EPI, HD, Quad>(A, lda, B, ldb, M, N, K, tiles_n, ep, s, splits);
  return launch_cfg<T, EPI, HD, Big>(A, lda, B, ldb, M, N, K, tiles_n, ep, s, splits);
}

// ---------------------------------------------------------------- split-K reductions

constexpr int kRedThreads = 256;

// x[row][c..c+3] += part[0] + part[1] + ... (in this order)
__global__ __launch_bounds__(kRedThreads) void splitk_resid_kernel(const float* __restrict__ part, int splits,
                                                                   int M, int N, int np, float* __restrict__ x,
                                                                   int ldx) {
  const int n4 = N >> 2;
  const int i = blockIdx.x * kRedThreads + threadIdx.x;
  if (i >= M * n4) return;
  const int row = i / n4, c = (i - row * n4) * 4;
  f32x4 acc = *reinterpret_cast<const f32x4*>(x + size_t(row) * ldx + c);
  auto pr = [&](int p) { return *reinterpret_cast<const f32x4*>(part + (size_t(p) * M + row) * np + c); };
  int p = 0;
  for (; p + 8 <= splits; p += 8) {   // eight loads in flight, added in order
    f32x4 a[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) a[q] = pr(p + q);
#pragma unroll
    for (int q = 0; q < 8; ++q) acc += a[q];
  }
  for (; p < splits; ++p) acc += pr(p);
  *reinterpret_cast<f32x4*>(x + size_t(row) * ldx + c) = acc;
}

// out[row][j..j+3] = silu(g) * u; gate j sits at partial column
// (j / 128) * 256 + ((j % 128) / 64) * 128 + j % 64, its up partner 64 further
template <typename T>
__global__ __launch_bounds__(kRedThreads) void splitk_swiglu_kernel(const float* __restrict__ part, int splits,
                                                                    int M, int F, int np, T* __restrict__ out) {
  const int f4 = F >> 2;
  const int i = blockIdx.x * kRedThreads + threadIdx.x;
  if (i >= M * f4) return;
  const int row = i / f4, j = (i - row * f4) * 4;
  const int gc = (j >> 7) * 256 + ((j & 127) >> 6) * 128 + (j & 63);
  f32x4 g = f32x4{0.f, 0.f, 0.f, 0.f}, u = g;
  const float* src = part + size_t(row) * np + gc;
  const size_t stride = size_t(M) * np;
  int p = 0;
  for (; p + 2 <= splits; p += 2) {
    const f32x4 g0 = *reinterpret_cast<const f32x4*>(src + p * stride),
                u0 = *reinterpret_cast<const f32x4*>(src + p * stride + 64),
                g1 = *reinterpret_cast<const f32x4*>(src + (p + 1) * stride),
                u1 = *reinterpret_cast<const f32x4*>(src + (p + 1) * stride + 64);
    g += g0;
    u += u0;
    g += g1;
    u += u1;
  }
  for (; p < splits; ++p) {
    g += *reinterpret_cast<const f32x4*>(src + p * stride);
    u += *reinterpret_cast<const f32x4*>(src + p * stride + 64);
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) store_f(out + size_t(row) * F + j + e, g[e] / (1.0f + __expf(-g[e])) * u[e]);
}


// four consecutive values stored at once (p 8-byte aligned for bf16, 16 for fp32)
__device__ __forceinline__ void store4(bf16_t* p, f32x4 v) {
  *reinterpret_cast<u32x2*>(p) = u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
}
__device__ __forceinline__ void store4(float* p, f32x4 v) { *reinterpret_cast<f32x4*>(p) = v; }
__device__ __forceinline__ void store4_vt(bf16_t* p, f32x4 v) {
  *reinterpret_cast<u32x2*>(p) = u32x2{pack_vt2(v[0], v[1]), pack_vt2(v[2], v[3])};
}
__device__ __forceinline__ void store4_vt(float* p, f32x4 v) { *reinterpret_cast<f32x4*>(p) = v; }

// Q and K: one thread per (row, q or k, head, 4 dims < HD/2): sums the two
// partner groups over the parts in order, rotates them and writes both to
// the head-major layout, 16-byte partial loads and 4-value stores
template <typename T, int HD>
__device__ __forceinline__ void splitk_qk(const float* __restrict__ part, int splits, int M, int np,
                                          const QkvOut& o, int blk) {
  constexpr int half = HD / 2, q4 = half / 4;
  const int d = o.d, per_row = d / 4;   // (q, k) x heads x half / 4
  const int i = blk * kRedThreads + threadIdx.x;
  if (i >= M * per_row) return;
  const int row = i / per_row, p = i - row * per_row;
  const int which = p / (per_row / 2), rest = p - which * (per_row / 2);
  const int h = rest / q4, dim = (rest - h * q4) * 4;
  const float* src = part + size_t(row) * np + which * d + h * HD + dim;
  const size_t stride = size_t(M) * np;
  f32x4 x1 = f32x4{0.f, 0.f, 0.f, 0.f}, x2 = x1;
  int s = 0;
  for (; s + 2 <= splits; s += 2) {
    const f32x4 a0 = *reinterpret_cast<const f32x4*>(src + s * stride),
                b0 = *reinterpret_cast<const f32x4*>(src + s * stride + half),
                a1 = *reinterpret_cast<const f32x4*>(src + (s + 1) * stride),
                b1 = *reinterpret_cast<const f32x4*>(src + (s + 1) * stride + half);
    x1 += a0;
    x2 += b0;
    x1 += a1;
    x2 += b1;
  }
  for (; s < splits; ++s) {
    x1 += *reinterpret_cast<const f32x4*>(src + s * stride);
    x2 += *reinterpret_cast<const f32x4*>(src + s * stride + half);
  }
  const float4* cs4 = reinterpret_cast<const float4*>(o.rope + size_t(qkv_pos(o, row)) * half + dim);
  const float4 c01 = cs4[0], c23 = cs4[1];   // (cos, sin) of dims dim .. dim + 3
  const float cs_c[4] = {c01.x, c01.z, c23.x, c23.z}, cs_s[4] = {c01.y, c01.w, c23.y, c23.w};
  f32x4 y1, y2;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    y1[e] = x1[e] * cs_c[e] - x2[e] * cs_s[e];
    y2[e] = x1[e] * cs_s[e] + x2[e] * cs_c[e];
  }
  const int b = row / o.seq, sp = row - b * o.seq;
  T* dst = static_cast<T*>(which == 0 ? o.q : o.k) + (size_t(b * o.H + h) * o.seq + sp) * HD + dim;
  store4(dst, y1);
  store4(dst + half, y2);
}

// V: 16-row x 64-column tiles transposed through LDS so that both the partial
// reads (16 bytes along a row) and the V^T writes (4 positions of one head
// dim) are contiguous
template <typename T>
__device__ __forceinline__ void splitk_v(const float* __restrict__ part, int splits, int M, int np, const QkvOut& o,
                                         int bx, int by, float (&tile)[16][65]) {
  const int c0 = bx * 64, r0 = by * 16, d = o.d;
  {
    const int r = threadIdx.x >> 4, c = (threadIdx.x & 15) * 4, row = r0 + r, col = c0 + c;
    f32x4 v = f32x4{0.f, 0.f, 0.f, 0.f};
    if (row < M && col < d) {   // d % 4 == 0: the 4 columns are in range together
      const float* src = part + size_t(row) * np + 2 * d + col;
      const size_t stride = size_t(M) * np;
      int p = 0;
      for (; p + 4 <= splits; p += 4) {
        const f32x4 a0 = *reinterpret_cast<const f32x4*>(src + p * stride),
                    a1 = *reinterpret_cast<const f32x4*>(src + (p + 1) * stride),
                    a2 = *reinterpret_cast<const f32x4*>(src + (p + 2) * stride),
                    a3 = *reinterpret_cast<const f32x4*>(src + (p + 3) * stride);
        v += a0;
        v += a1;
        v += a2;
        v += a3;
      }
      for (; p < splits; ++p) v += *reinterpret_cast<const f32x4*>(src + p * stride);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) tile[r][c + e] = v[e];
  }
  __syncthreads();
  const int c = threadIdx.x >> 2, rg = (threadIdx.x & 3) * 4, col = c0 + c, row = r0 + rg;
  if (col >= d || row >= M) return;
  const int b = row / o.seq, sp = row - b * o.seq, h = col / o.hd, dim = col - h * o.hd;
  T* dst = static_cast<T*>(o.vt) + (size_t(b * o.H + h) * o.hd + dim) * o.vt_ld + sp;
  // 4 positions of one sequence, aligned
  if ((o.seq % 4) == 0 && row + 3 < M && (reinterpret_cast<uintptr_t>(dst) & (4 * sizeof(T) - 1)) == 0) {
    store4_vt(dst, f32x4{tile[rg][c], tile[rg + 1][c], tile[rg + 2][c], tile[rg + 3][c]});
  } else {
    for (int e = 0; e < 4 && row + e < M; ++e) {
      const int bi = (row + e) / o.seq, si = (row + e) - bi * o.seq;
      store_vt(static_cast<T*>(o.vt) + (size_t(bi * o.H + h) * o.hd + dim) * o.vt_ld + si, tile[rg + e][c]);
    }
  }
}

// the QKV split-K sums in one launch: blocks 0 .. n_qk - 1 take Q and K, the
// rest the V tiles (d / 64 column tiles by M / 16 row tiles)
template <typename T, int HD>
__global__ __launch_bounds__(kRedThreads) void splitk_qkv_kernel(const float* __restrict__ part, int splits, int M,
                                                                 int np, QkvOut o, int n_qk) {
  __shared__ float tile[16][65];
  const int blk = blockIdx.x;
  if (blk < n_qk) {
    splitk_qk<T, HD>(part, splits, M, np, o, blk);
  } else {
    const int v = blk - n_qk, nvx = cdiv(o.d, 64);
    splitk_v<T>(part, splits, M, np, o, v % nvx, v / nvx, tile);
  }
}

}  // namespace

hipError_t splitk_add(const SplitK& sk, int M, int N, float* X, int ldx, hipStream_t s) {
  if (N % 4 || ldx % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(splitk_resid_kernel, dim3(cdiv(M * (N / 4), kRedThreads)), dim3(kRedThreads), 0, s, sk.part,
                     sk.splits, M, N, cdiv(N, kBN) * kBN, X, ldx);
  return hipGetLastError();
}

int gemm_splits(int kind, int M, int N, int K, int dtype) {
  // workgroups that fill the 256 CUs: one Big, Mid or Quad workgroup per CU, two Small ones
  const int bm = tile_rows(kind, M, N, K);
  const int tiles_n = kind == GEMM_KIND_GATEUP ? cdiv(N / 2, 128)
                      : kind == GEMM_KIND_QKV && qkv_mid_parts(M, N) ? N / Mid::BN
                                                                       : cdiv(N, kBN);
  const int tiles = cdiv(M, bm) * tiles_n, full = bm == Small::BM ? 512 : 256;
  const int stages = K / (dtype ? 64 : 32);   // 128-byte K stages
  if (tiles >= full * 5 / 8 || stages < 2) return 1;
  const int parts = std::max(1, std::min(full / tiles, stages / 4));
  // a multiple of 8 or a power of two, so that map_split_tile gives each
  // XCD whole parts (or an even share of one)
  if (parts >= 8) return parts / 8 * 8;
  int p2 = 1;
  while (p2 * 2 <= parts) p2 *= 2;
  return p2;
}

size_t gemm_partial_bytes(int M, int tiles_n, int splits) {
  return splits > 1 ? size_t(splits) * M * tiles_n * kBN * sizeof(float) : 0;
}

hipError_t gemm_resid(int dtype, const void* A, int lda, const void* B, int ldb, int M, int N, int K, float* X,
                      int ldx, hipStream_t s, const SplitK* sk) {
  if (N % 4 || ldx % 4 || reinterpret_cast<uintptr_t>(X) % 16) return hipErrorInvalidValue;   // 16-byte x accesses
  EpiParams ep{};
  ep.x = X;
  ep.ldx = ldx;
  const int tn = cdiv(N, kBN);
  const int bm = tile_rows(GEMM_KIND_RESID, M, N, K);
  if (sk && sk->splits > 1) {
    ep.part = sk->part;
    ep.np = tn * kBN;
    hipError_t e = dtype ? launch<bf16_t, EPI_PART>(bm, A, lda, B, ldb, M, N, K, tn, ep, s, sk->splits)
                         : launch<float, EPI_PART>(bm, A, lda, B, ldb, M, N, K, tn, ep, s, sk->splits);
    if (e != hipSuccess || sk->defer) return e;
    return splitk_add(*sk, M, N, X, ldx, s);
  }
  return dtype ? launch<bf16_t, EPI_RESID>(bm, A, lda, B, ldb, M, N, K, tn, ep, s)
               : launch<float, EPI_RESID>(bm, A, lda, B, ldb, M, N, K, tn, ep, s);
}

hipError_t gemm_swiglu(int dtype, const void* A, int lda, const void* Wgu, int M, int F, int K, void* out,
                       hipStream_t s, const SplitK* sk) {
  EpiParams ep{};
  ep.out = out;
  ep.F = F;
  const int bm = tile_rows(GEMM_KIND_GATEUP, M, 2 * F, K);
  if (!(sk && sk->splits > 1) && M > 256 && M <= 512 && bm == Big::BM) {
    const int tm = cdiv(F, Mid::BN / 2);
    return dtype ? launch_cfg<bf16_t, EPI_SWIGLU, 0, Mid>(A, lda, Wgu, K, M, 2 * F, K, tm, ep, s, 1)
                 : launch_cfg<float, EPI_SWIGLU, 0, Mid>(A, lda, Wgu, K, M, 2 * F, K, tm, ep, s, 1);
  }
  const int tn = cdiv(F, 128);
  if (sk && sk->splits > 1) {
    if (F % 4) return hipErrorInvalidValue;
    ep.part = sk->part;
    ep.np = tn * kBN;
    hipError_t e = dtype ? launch<bf16_t, EPI_PART_GU>(bm, A, lda, Wgu, K, M, 2 * F, K, tn, ep, s, sk->splits)
                         : launch<float, EPI_PART_GU>(bm, A, lda, Wgu, K, M, 2 * F, K, tn, ep, s, sk->splits);
    if (e != hipSuccess) return e;
    const dim3 g(cdiv(M * (F / 4), kRedThreads));
    if (dtype)
      hipLaunchKernelGGL(splitk_swiglu_kernel<bf16_t>, g, dim3(kRedThreads), 0, s, sk->part, sk->splits, M, F, ep.np,
                         static_cast<bf16_t*>(out));
    else
      hipLaunchKernelGGL(splitk_swiglu_kernel<float>, g, dim3(kRedThreads), 0, s, sk->part, sk->splits, M, F, ep.np,
                         static_cast<float*>(out));
    return hipGetLastError();
  }
  if (bm == Big::BM) {
    // 256 x 256 tiles, one persistent workgroup per CU
    const int stage_k = dtype ? 2 * TileMma<bf16_t, Big::BM, Big::BN, Big::WM, Big::WN>::kKPerStage
                              : 2 * TileMma<float, Big::BM, Big::BN, Big::WM, Big::WN>::kKPerStage;
    if (K <= 0 || K % stage_k) return hipErrorInvalidValue;
    const int tiles_m = cdiv(M, Big::BM), tiles = tiles_m * tn;
    const int grid = std::min(tiles, device_cus());
    if (dtype)
      hipLaunchKernelGGL((gemm_swiglu_persist_kernel<bf16_t, Big>), dim3(grid), dim3(Big::kThreads), 0, s,
                         static_cast<const bf16_t*>(A), lda, static_cast<const bf16_t*>(Wgu), M, K, tiles_m, tn, ep);
    else
      hipLaunchKernelGGL((gemm_swiglu_persist_kernel<float, Big>), dim3(grid), dim3(Big::kThreads), 0, s,
                         static_cast<const float*>(A), lda, static_cast<const float*>(Wgu), M, K, tiles_m, tn, ep);
    return hipGetLastError();
  }
  return dtype ? launch<bf16_t, EPI_SWIGLU>(bm, A, lda, Wgu, K, M, 2 * F, K, tn, ep, s)
               : launch<float, EPI_SWIGLU>(bm, A, lda, Wgu, K, M, 2 * F, K, tn, ep, s);
}

namespace {

template <typename T>
hipError_t qkv_split(const void* A, int lda, const void* Wqkv, int M, int K, const QkvOut& o, hipStream_t s,
                     const SplitK& sk) {
  if (o.d % 8) return hipErrorInvalidValue;   // the reduction takes groups of 4 dims of every head half
  EpiParams ep{};
  ep.qkv = o;
  const int N = 3 * o.d, tn = cdiv(N, kBN);
  ep.part = sk.part;
  ep.np = tn * kBN;   // the partial layout does not depend on the tiling
  hipError_t e = qkv_mid_parts(M, N)
                     ? launch_cfg<T, EPI_PART, 0, Mid>(A, lda, Wqkv, K, M, N, K, N / Mid::BN, ep, s, sk.splits)
                     : launch<T, EPI_PART>(tile_rows(GEMM_KIND_QKV, M, N, K), A, lda, Wqkv, K, M, N, K, tn, ep, s,
                                           sk.splits);
  if (e != hipSuccess) return e;
  const int n_qk = cdiv(M * (o.d / 4), kRedThreads), n_v = cdiv(o.d, 64) * cdiv(M, 16);
  if (o.hd == 128)
    hipLaunchKernelGGL((splitk_qkv_kernel<T, 128>), dim3(n_qk + n_v), dim3(kRedThreads), 0, s, sk.part, sk.splits,
                       M, ep.np, o, n_qk);
  else
    hipLaunchKernelGGL((splitk_qkv_kernel<T, 64>), dim3(n_qk + n_v), dim3(kRedThreads), 0, s, sk.part, sk.splits,
                       M, ep.np, o, n_qk);
  return hipGetLastError();
}

}  // namespace

hipError_t gemm_qkv(int dtype, const void* A, int lda, const void* Wqkv, int M, int K, const QkvOut& o,
                    hipStream_t s, const SplitK* sk) {
  if (sk && sk->splits > 1)
    return dtype ? qkv_split<bf16_t>(A, lda, Wqkv, M, K, o, s, *sk) : qkv_split<float>(A, lda, Wqkv, M, K, o, s, *sk);
  EpiParams ep{};
  ep.qkv = o;
  const int N = 3 * o.d;
  const int tn = cdiv(N, kBN);
  const int bm = tile_rows(GEMM_KIND_QKV, M, N, K);
  if (o.hd == 128)
    return dtype ? launch<bf16_t, EPI_QKV, 128>(bm, A, lda, Wqkv, K, M, N, K, tn, ep, s)
                 : launch<float, EPI_QKV, 128>(bm, A, lda, Wqkv, K, M, N, K, tn, ep, s);
  return dtype ? launch<bf16_t, EPI_QKV, 64>(bm, A, lda, Wqkv, K, M, N, K, tn, ep, s)
               : launch<float, EPI_QKV, 64>(bm, A, lda, Wqkv, K, M, N, K, tn, ep, s);
}

}  // namespace dllm
