// Full non-causal softmax attention, softmax(q k^T / sqrt(hd)) v over every
// key of the sequence, optionally preceded by the keys of a cached prefix
// (shared by all sequences of the batch).
//
// A workgroup of 4 waves takes 128 queries of one (sequence, head); each
// wave owns 32 queries, two workgroups share a CU.  Short sequences (at most
// 64 queries, e.g. a block recomputed over a cached prefix), and launches
// whose 128-query workgroups would leave CUs idle (a single sequence of
// 512), take 32 queries per workgroup instead: wave w owns the 16 queries of
// block w % 2 and the keys of half w / 2 of every tile, and the two halves'
// softmax states are merged at the end; when even that layout leaves most
// CUs idle (one block of 32 over a long cached prefix: 32 workgroups), each
// sequence's key tiles are also split into ranges, one workgroup each, and a
// merge kernel combines the ranges' states in a fixed order.  Keys stream
// through a two-slot LDS ring in tiles of 64 (K rows and V^T columns), copied
// from global memory straight into LDS with buffer_load ... lds one tile
// ahead.
// Scores are computed transposed, S^T = K Q^T, so in the MFMA output layout
// every lane holds one query's scores for 4 keys per 16-key block: the
// online-softmax max/sum and the output rescale stay per lane, and the
// probabilities feed the P V product (computed as O^T = V^T P^T) directly as
// MFMA operands without an LDS round trip.  bf16 models keep V^T in IEEE
// binary16 (written so by the QKV projection), and P V runs on fp16 MFMAs.
#include <algorithm>

#include "kernels.h"
#include "common.h"
#include "mainloop.h"

namespace dllm {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * kWave;
constexpr int kQW = 32;             // queries per wave
constexpr int kQT = kWaves * kQW;   // queries per workgroup
constexpr int kKT = 64;             // keys per tile
constexpr int kSplitMaxQ = 64;      // sequences of at most this many queries take the split layout
constexpr int kSplitMaxWg = 256;    // so do launches whose 128-query layout has fewer workgroups than this
// Key split of the split layout: launches of fewer than kKvMinWg workgroups
// split every sequence's key tiles into up to kKvMaxSplits ranges of at least
// two tiles (one-tile ranges measured slower: each range pays its own fill
// and the merge grows), one workgroup each, whose partial states a merge
// kernel combines
constexpr int kKvMinWg = 128;
constexpr int kKvMaxSplits = 16;
constexpr int kKvTargetWg = 512;
// floats per partial record: HD output values, m, l, padding to 16 bytes
constexpr int kv_rec(int hd) { return hd + 4; }

// key ranges of a split-layout launch of wg workgroups over n_tiles key tiles
int kv_splits_of(int wg, int n_tiles) {
  if (wg >= kKvMinWg) return 1;
  return std::max(1, std::min({kKvMaxSplits, n_tiles / 2, kKvTargetWg / wg}));
}

template <typename T, int HD>
struct AttnCfg {
  static constexpr int E = Elem<T>::per_chunk;             // elements per 16-byte chunk
  static constexpr int CK = HD * Elem<T>::bytes / 16;      // chunks per K row
  static constexpr int CV = kKT * Elem<T>::bytes / 16;     // chunks per V^T row (64 keys)
  static constexpr int KB = kKT * CK * 16;                 // K tile bytes
  static constexpr int VB = HD * CV * 16;                  // V^T tile bytes
  static constexpr int STAGE = KB + VB;
  static constexpr int RK = 64 / CK;                       // K rows per load instruction (1 KB)
  static constexpr int RV = 64 / CV;                       // V^T rows per load instruction
  static constexpr int IK = kKT * CK / 64 / kWaves;        // K load instructions per wave per tile
  static constexpr int IV = HD * CV / 64 / kWaves;         // V^T load instructions per wave per tile
  static constexpr int NDB = HD / 16;                      // 16-row dim blocks of O^T
  static constexpr int QSTEPS = CK / 4;                    // MFMA k-steps over head_dim
  static_assert(CK >= 8 && CV >= 8, "rows of at least 8 chunks (swizzle)");
  static_assert(IK * kWaves * 64 == kKT * CK && IV * kWaves * 64 == HD * CV, "tile split");
};

// row r, chunk c of a tile stored with rows of `row_bytes`: chunk slot c ^ (r % 8)
__device__ __forceinline__ int swz(int r, int c, int row_bytes) { return r * row_bytes + ((c ^ (r & 7)) << 4); }

// K tiles (bf16): chunk c of key row r in slot c ^ kswz(r).  An S^T block
// reads the 16 rows 8 q + 4 kk + j (q, j < 4, see key_of); this swizzle maps
// them to 16 distinct slots with 16 chunks per row (8 with 8), so the 16
// lanes of a read touch distinct LDS banks.  fp32 tiles read 16 consecutive
// rows: r % 8, as for V^T.
// max / sum over lanes l, l ^ 16, l ^ 32, l ^ 48 (the four 16-lane groups
// that hold one query's scores): two permlane swaps on the vector ALU
// instead of two LDS permutes
__device__ __forceinline__ float group4_max(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float u = __uint_as_float(a[0]), v = __uint_as_float(a[1]);
  const float m = u > v ? u : v;
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(m), __float_as_uint(m), false, false);
  const float p = __uint_as_float(b[0]), q = __uint_as_float(b[1]);
  return p > q ? p : q;
}
__device__ __forceinline__ float group4_sum(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float m = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(m), __float_as_uint(m), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

template <typename T, int CK>
__device__ __forceinline__ int kswz(int r) {
  if constexpr (Elem<T>::per_chunk == 8)
    return CK >= 16 ? ((r & 3) | (((r >> 3) & 3) << 2)) : ((r & 3) | (((r >> 3) & 1) << 2));
  else
    return r & 7;
}

// kv_splits > 1 (split layout only): blockIdx.x = query block * kv_splits +
// key range; the workgroup writes its unnormalised output and (m, l) to
// a.kv_part instead of the normalised output
template <typename T, int HD, bool kPacked, bool kSplit>
__global__ __launch_bounds__(kThreads, 2) void attn_kernel(AttnArgs a, float qk_scale_log2, int kv_splits) {
  using C = AttnCfg<T, HD>;
  static_assert(!(kPacked && kSplit), "the split layout serves unpacked sequences");
  constexpr int NQB = kSplit ? 1 : 2;   // 16-query blocks per wave
  constexpr int NH = kSplit ? 1 : 2;    // 32-key halves of a tile per wave
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * C::STAGE];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int fr = lane & 15, g = lane >> 4;
  const int b = blockIdx.z, h = blockIdx.y;
  // split: the wave's query block and key half
  const int qsel = kSplit ? (wave & 1) : 0, hsel = kSplit ? (wave >> 1) : 0;
  const int qblk = kSplit ? int(blockIdx.x) / kv_splits : int(blockIdx.x);
  const int q0 = kSplit ? qblk * kQW + 16 * qsel : qblk * kQT + wave * kQW;
  const size_t bh = size_t(b) * a.H + h;

  const T* Q = static_cast<const T*>(a.q) + bh * a.Sq * HD;
  const uint8_t* Ko = reinterpret_cast<const uint8_t*>(static_cast<const T*>(a.k) + bh * a.Sq * HD);
  const uint8_t* Vo = reinterpret_cast<const uint8_t*>(static_cast<const T*>(a.vt) + bh * HD * a.vt_ld);
  const uint8_t* Kp = a.kp ? reinterpret_cast<const uint8_t*>(static_cast<const T*>(a.kp) + size_t(h) * a.p_cap * HD)
                           : nullptr;
  const uint8_t* Vp =
      a.kp ? reinterpret_cast<const uint8_t*>(static_cast<const T*>(a.vpt) + size_t(h) * HD * a.p_cap) : nullptr;
  const int n_pt = a.kp ? cdiv(a.p_len, kKT) : 0;
  // Packed lookahead (pack_B > 0): the shared rows 0 .. S-1 attend to each
  // other only; a branch block's rows attend to the shared rows outside the
  // block they stand in for (b0 .. b0+pack_B-1) and to their own block.
  // Phase 1 tiles cover keys 0 .. S-1, phase 2 tiles the branch blocks that
  // hold this workgroup's branch queries, each block on tiles of its own.
  constexpr bool packed = kPacked;   // a.pack_B > 0
  const int S = packed ? a.pack_S : a.Sq;
  const int n_ot = cdiv(S, kKT);
  int jb0 = 0, tpb = 1, n_bt = 0;
  if (packed) {
    const int qlo = max(int(blockIdx.x) * kQT, S), qhi = min(int(blockIdx.x) * kQT + kQT, a.Sq);
    if (qlo < qhi) {
      jb0 = (qlo - S) / a.pack_B;
      tpb = cdiv(a.pack_B, kKT);
      n_bt = ((qhi - 1 - S) / a.pack_B - jb0 + 1) * tpb;
    }
  }
  const int n_tiles = n_pt + n_ot + n_bt;
  // this workgroup's key tiles tb .. te - 1 (a key range of the split layout)
  int tb = 0, te = n_tiles;
  if constexpr (kSplit) {
    const int ks = int(blockIdx.x) % kv_splits;
    tb = ks * n_tiles / kv_splits;
    te = (ks + 1) * n_tiles / kv_splits;
  }
  // branch of each of this lane's two query columns (-1: a shared row)
  int qbr[2];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int q = q0 + qb * 16 + fr;
    qbr[qb] = packed && q >= S ? (q - S) / a.pack_B : -1;
  }

  // Q fragments (B operand of S^T = K Q^T): query q0 + 16 qb + fr, chunk 4 step + g
  u32x4 qf[NQB][C::QSTEPS];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    const int q = min(q0 + qb * 16 + fr, a.Sq - 1);
#pragma unroll
    for (int st = 0; st < C::QSTEPS; ++st)
      qf[qb][st] = *reinterpret_cast<const u32x4*>(reinterpret_cast<const uint8_t*>(Q + size_t(q) * HD) +
                                                   (4 * st + g) * 16);
  }

  // Key (within the tile) of row r of S^T block kk in half h.  bf16: the
  // rows of a 32-key half are gathered so that S^T output element i of lane
  // group g in block kk is key 32 h + 8 g + 4 kk + i: each lane's 8
  // probabilities of the half are 8 consecutive keys, i.e. one 16-byte chunk
  // of a V^T row (the P V operand).  fp32 (4 keys per chunk): plain order.
  auto key_of = [](int h, int kk, int r) {
    if constexpr (Elem<T>::per_chunk == 8) return 32 * h + 8 * (r >> 2) + 4 * kk + (r & 3);
    else return 32 * h + 16 * kk + r;
  };
  const uint32_t lds0 = lds_address(smem);
  // key range of tile t: source, first key, number of valid keys of the source, V^T row pitch
  struct Src {
    const uint8_t* k;
    const uint8_t* v;
    int k0, nk, ld;
    int branch;   // phase-2 tile: the branch block it covers; -1 otherwise
    bool prefix;  // a tile of the cached prefix (visible to every query)
  };
  auto src = [&](int t) -> Src {
    if (t < n_pt) return Src{Kp, Vp, t * kKT, a.p_len, a.p_cap, -1, true};
    if (t < n_pt + n_ot) return Src{Ko, Vo, (t - n_pt) * kKT, S, a.vt_ld, -1, false};
    const int u = t - n_pt - n_ot, j = jb0 + u / tpb;
    return Src{Ko, Vo, S + j * a.pack_B + (u % tpb) * kKT, S + (j + 1) * a.pack_B, a.vt_ld, j, false};
  };
  // Copy tile t into ring slot `slot`.  Lane l of a load instruction fills
  // row l / C, slot l % C of its block and fetches the chunk the swizzle
  // assigns there.  Rows past the last valid key read the last valid row and
  // V^T chunks past the row pitch read the row's last chunk: every address
  // stays inside the source, and those keys are masked (K) or zeroed (V^T).
  auto issue = [&](int t, int slot) {
    const Src s = src(t);
    const rsrc_t rk = buffer_rsrc(s.k), rv = buffer_rsrc(s.v);
    const uint32_t base = lds0 + slot * C::STAGE;
#pragma unroll
    for (int i = 0; i < C::IK; ++i) {
      const int grp = wave * C::IK + i;
      const int r = grp * C::RK + lane / C::CK, c = (lane % C::CK) ^ kswz<T, C::CK>(r);
      const int key = min(s.k0 + r, s.nk - 1);
      lds_dma16(rk, uint32_t(key) * (HD * Elem<T>::bytes) + c * 16, 0, base + grp * 1024);
    }
#pragma unroll
    for (int i = 0; i < C::IV; ++i) {
      const int grp = wave * C::IV + i;
      const int r = grp * C::RV + lane / C::CV, c = (lane % C::CV) ^ (r & 7);
      const int key = min(s.k0 + c * C::E, s.ld - C::E);
      lds_dma16(rv, (uint32_t(r) * s.ld + key) * Elem<T>::bytes, 0, base + C::KB + grp * 1024);
    }
  };
  auto ragged = [&](int t) {
    const Src s = src(t);
    return s.nk - s.k0 < kKT;
  };
  // zero the V^T values of keys >= nk in a ragged tile (after it has landed)
  auto zero_tail = [&](int t, int slot) {
    const Src s = src(t);
    const int valid = s.nk - s.k0;
    uint8_t* sv = smem + slot * C::STAGE + C::KB;
    for (int q = tid; q < HD * C::CV; q += kThreads) {
      const int r = q / C::CV, c = q % C::CV, e0 = c * C::E;
      if (e0 + C::E <= valid) continue;
      u32x4* p = reinterpret_cast<u32x4*>(sv + swz(r, c, C::CV * 16));
      if (e0 >= valid) {
        *p = u32x4{0u, 0u, 0u, 0u};
      } else {
        T* el = reinterpret_cast<T*>(p);
        for (int e = valid - e0; e < C::E; ++e) el[e] = T{};
      }
    }
  };

  f32x4 o[C::NDB][NQB];
#pragma unroll
  for (int db = 0; db < C::NDB; ++db)
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) o[db][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float mrun[NQB], lrun[NQB];   // exponent reference (log2 units) and this lane's part of the sum
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    mrun[qb] = -INFINITY;
    lrun[qb] = 0.f;
  }

  issue(tb, 0);
  wait_vmcnt<0>();
  __syncthreads();
  if (ragged(tb)) {
    zero_tail(tb, 0);
    __syncthreads();
  }
  for (int t = tb; t < te; ++t) {
    const bool more = t + 1 < te;
    const int slot = (t - tb) & 1;
    if (more) issue(t + 1, slot ^ 1);   // that slot was last read before the previous barrier
    const uint8_t* s = smem + slot * C::STAGE;
    const uint8_t* sv = s + C::KB;
    const Src sr = src(t);
    const int k0 = sr.k0, nk = sr.nk;
    // does the packing mask keys of this tile?  phase 2 always; phase 1 where
    // the tile meets the stood-in block and the workgroup has branch queries;
    // never a tile of the cached prefix
    const bool pmask = packed && !sr.prefix &&
                       (sr.branch >= 0 || (n_bt > 0 && k0 < a.pack_b0 + a.pack_B && k0 + kKT > a.pack_b0));

    // the tile's 64 keys in two halves of 32: S^T, online softmax and P V per half
#pragma unroll
    for (int hh = 0; hh < NH; ++hh) {
      const int half = kSplit ? hsel : hh;
      // S^T block (key block 2 half + kk, query block qb)
      f32x4 sc[2][NQB];
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb) sc[kk][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int st = 0; st < C::QSTEPS; ++st) {
          const int kr = key_of(half, kk, fr);
          const u32x4 kf = *reinterpret_cast<const u32x4*>(s + kr * (C::CK * 16) + (((4 * st + g) ^ kswz<T, C::CK>(kr)) << 4));
#pragma unroll
          for (int qb = 0; qb < NQB; ++qb) Mfma<T>::run(sc[kk][qb], kf, qf[qb][st]);
        }
      }
      // online softmax per query column (this lane's query q0 + 16 qb + fr)
      float p[2][NQB][4];
      float alpha[NQB];
      const bool full = !pmask && k0 + 32 * half + 32 <= nk;   // every key of this half is valid
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb) {
        float mt = -INFINITY;
        if (full) {   // wave-uniform: no key of this half is masked
#pragma unroll
          for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              p[kk][qb][i] = sc[kk][qb][i];
              mt = fmaxf(mt, sc[kk][qb][i]);
            }
        } else {
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int key = k0 + key_of(half, kk, 4 * g + i);
            bool ok = key < nk;
            if (pmask)
              ok = ok && (sr.branch >= 0 ? qbr[qb] == sr.branch
                                         : (qbr[qb] < 0 || key < a.pack_b0 || key >= a.pack_b0 + a.pack_B));
            const float v = ok ? sc[kk][qb][i] : -INFINITY;
            p[kk][qb][i] = v;
            mt = fmaxf(mt, v);
          }
        }
        mt = group4_max(mt);
        // The exponent reference moves only when a score exceeds it by more
        // than 8 (log2 units): probabilities stay below 2^8, o and l share the
        // reference so o / l is unchanged, and the accumulators are rescaled
        // rarely instead of at nearly every new maximum.
        const float mcand = mt * qk_scale_log2;
        const float mnew = mcand > mrun[qb] + 8.f ? mcand : mrun[qb];
        // packed (a branch query) or split (the second key half): a tile can
        // mask every key a wave sees before it has seen any; the reference
        // stays -inf and the exponents use 0, giving 0 instead of NaN
        float mref = mnew;
        if constexpr (kPacked || kSplit) mref = mnew == -INFINITY ? 0.f : mnew;
        alpha[qb] = __builtin_amdgcn_exp2f(mrun[qb] - mref);
        mrun[qb] = mnew;
        float ls = 0.f;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float e = __builtin_amdgcn_exp2f(fmaf(p[kk][qb][i], qk_scale_log2, -mref));
            p[kk][qb][i] = e;
            ls += e;
          }
        lrun[qb] = lrun[qb] * alpha[qb] + ls;
      }
      // rescale the accumulators only when some query of the wave has a new maximum
      bool moved = false;
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb) moved = moved || alpha[qb] != 1.f;
      if (__any(moved)) {
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
          for (int db = 0; db < C::NDB; ++db) o[db][qb] *= alpha[qb];
      }
      // O^T += V^T P^T over keys 32 half .. 32 half + 31
      if constexpr (Elem<T>::per_chunk == 8) {
        // P and V^T in IEEE binary16 (11 significant bits, probabilities
        // below 2^8 by the lazy reference), one fp16 MFMA per block, where
        // bf16 weights alone would add an error as large as the bf16 rounding
        // of the output over a thousand keys.  The split layout (launches
        // that leave CUs idle, and short blocks over a cached prefix) adds a
        // second MFMA on lo = fp16(p - hi), about 22 significant bits: it
        // costs little where the chip is not full.
        constexpr bool kPairP = kSplit;
        u32x4 pb[NQB], pl[NQB];
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const int kk = w >> 1, i0 = 2 * (w & 1);
            const float a0 = p[kk][qb][i0], a1 = p[kk][qb][i0 + 1];
            pb[qb][w] = pack_f16x2(a0, a1);
            if constexpr (kPairP)
              pl[qb][w] = pack_f16x2(a0 - f16_lo(pb[qb][w]), a1 - f16_hi(pb[qb][w]));
          }
#pragma unroll
        for (int db = 0; db < C::NDB; ++db) {
          // this lane's 8 probabilities are keys 32 half + 8 g .. + 7 (see key_of)
          const u32x4 vf = *reinterpret_cast<const u32x4*>(sv + swz(db * 16 + fr, 4 * half + g, C::CV * 16));
#pragma unroll
          for (int qb = 0; qb < NQB; ++qb) {
            MfmaF16::run(o[db][qb], vf, pb[qb]);
            if constexpr (kPairP) MfmaF16::run(o[db][qb], vf, pl[qb]);
          }
        }
      } else {
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          u32x4 pb[NQB];
#pragma unroll
          for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
            for (int i = 0; i < 4; ++i) pb[qb][i] = __float_as_uint(p[kk][qb][i]);
#pragma unroll
          for (int db = 0; db < C::NDB; ++db) {
            const int r = db * 16 + fr;
            const int key = (2 * half + kk) * 16 + 4 * g;  // 4 fp32 keys = one chunk
            const u32x4 vf = *reinterpret_cast<const u32x4*>(sv + swz(r, key >> 2, C::CV * 16));
#pragma unroll
            for (int qb = 0; qb < NQB; ++qb) Mfma<T>::run(o[db][qb], vf, pb[qb]);
          }
        }
      }
    }
    wait_vmcnt<0>();
    __syncthreads();
    if (more && ragged(t + 1)) {
      zero_tail(t + 1, slot ^ 1);
      __syncthreads();
    }
  }

  if constexpr (kSplit) {
    // Merge the second key half's state into the first's, lane by lane (the
    // same lane of the two waves holds the same query and dims): the ring is
    // free after the loop's last barrier.  The first half always holds key 0,
    // so its reference is finite; a second half that saw no key has l = 0
    // and reference -inf, and weighs 0.
    constexpr int NV = C::NDB * 4 + 2;
    static_assert(2 * NV * 64 * 4 <= 2 * C::STAGE, "merge buffer inside the ring");
    float* xs = reinterpret_cast<float*>(smem) + qsel * NV * 64 + lane;
    if (hsel == 1) {
#pragma unroll
      for (int db = 0; db < C::NDB; ++db)
#pragma unroll
        for (int i = 0; i < 4; ++i) xs[(4 * db + i) * 64] = o[db][0][i];
      xs[(NV - 2) * 64] = mrun[0];
      xs[(NV - 1) * 64] = lrun[0];
    }
    __syncthreads();
    if (hsel == 1) return;
    const float mb = xs[(NV - 2) * 64], lb = xs[(NV - 1) * 64];
    const float m = fmaxf(mrun[0], mb);
    const float sa = __builtin_amdgcn_exp2f(mrun[0] - m), sb = __builtin_amdgcn_exp2f(mb - m);
#pragma unroll
    for (int db = 0; db < C::NDB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) o[db][0][i] = o[db][0][i] * sa + xs[(4 * db + i) * 64] * sb;
    lrun[0] = lrun[0] * sa + lb * sb;
    mrun[0] = m;
    if (kv_splits > 1) {
      // the key range's state: unnormalised output rows (this lane: dims
      // 16 db + 4 g + i of query q), the reference m (log2 units) and l
      const int q = q0 + fr;
      const float l = group4_sum(lrun[0]);
      if (q < a.Sq) {
        const int ks = int(blockIdx.x) % kv_splits;
        float* rec = a.kv_part + ((size_t(ks) * a.B * a.H + bh) * a.Sq + q) * kv_rec(HD);
#pragma unroll
        for (int db = 0; db < C::NDB; ++db)
          *reinterpret_cast<f32x4*>(rec + db * 16 + 4 * g) = o[db][0];
        if (g == 0) {
          rec[HD] = m;
          rec[HD + 1] = l;
        }
      }
      return;
    }
  }

  // normalise and store O[b * Sq + q][h * HD + dim]
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    const float l = group4_sum(lrun[qb]);
    const float inv = 1.0f / l;
    const int q = q0 + qb * 16 + fr;
    if (q >= a.Sq) continue;
    T* orow = static_cast<T*>(a.o) + (size_t(b) * a.Sq + q) * (size_t(a.H) * HD) + size_t(h) * HD;
#pragma unroll
    for (int db = 0; db < C::NDB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) store_f(orow + db * 16 + 4 * g + i, o[db][qb][i] * inv);
  }
}

// merge of the key ranges' partial states: out[b * Sq + q][h * HD + dim] =
// sum_s o_s 2^(m_s - m) / sum_s l_s 2^(m_s - m), m = max_s m_s, the ranges
// added in order; one workgroup of HD threads per (b, h, q)
template <typename T, int HD>
__global__ __launch_bounds__(HD) void attn_merge_kernel(AttnArgs a, int kv_splits) {
  const int q = blockIdx.x, h = blockIdx.y, b = blockIdx.z, dim = threadIdx.x;
  const size_t bh = size_t(b) * a.H + h, stride = size_t(a.B) * a.H * a.Sq * kv_rec(HD);
  const float* rec = a.kv_part + (bh * a.Sq + q) * kv_rec(HD);
  float m = -INFINITY;
  for (int ks = 0; ks < kv_splits; ++ks) m = fmaxf(m, rec[ks * stride + HD]);
  float o = 0.f, l = 0.f;
  for (int ks = 0; ks < kv_splits; ++ks) {
    const float w = __builtin_amdgcn_exp2f(rec[ks * stride + HD] - m);
    o += rec[ks * stride + dim] * w;
    l += rec[ks * stride + HD + 1] * w;
  }
  store_f(static_cast<T*>(a.o) + (size_t(b) * a.Sq + q) * (size_t(a.H) * HD) + size_t(h) * HD + dim, o / l);
}

template <typename T, int HD>
hipError_t launch_attn(const AttnArgs& a, hipStream_t s) {
  // the V^T copies read whole 16-byte chunks inside each row of pitch vt_ld / p_cap
  if (a.vt_ld < 8 || a.vt_ld % 8 || (a.kp && (a.p_cap < 8 || a.p_cap % 8))) return hipErrorInvalidValue;
  if (a.pack_B > 0 && (a.B != 1 || a.pack_S < 1 || a.pack_S > a.Sq || (a.Sq - a.pack_S) % a.pack_B ||
                       a.pack_b0 < 0 || a.pack_b0 + a.pack_B > a.pack_S))
    return hipErrorInvalidValue;
  const float scale = 1.4426950408889634f / sqrtf(float(HD));
  if (a.pack_B > 0) {
    hipLaunchKernelGGL((attn_kernel<T, HD, true, false>), dim3(cdiv(a.Sq, kQT), a.H, a.B), dim3(kThreads), 0, s, a,
                       scale, 1);
  } else if (a.Sq <= kSplitMaxQ || cdiv(a.Sq, kQT) * a.H * a.B < kSplitMaxWg) {
    const int wg = cdiv(a.Sq, kQW) * a.H * a.B;
    const int n_tiles = (a.kp ? cdiv(a.p_len, kKT) : 0) + cdiv(a.Sq, kKT);
    const int kv = a.kv_part ? kv_splits_of(wg, n_tiles) : 1;
    hipLaunchKernelGGL((attn_kernel<T, HD, false, true>), dim3(cdiv(a.Sq, kQW) * kv, a.H, a.B), dim3(kThreads), 0,
                       s, a, scale, kv);
    if (kv > 1) hipLaunchKernelGGL((attn_merge_kernel<T, HD>), dim3(a.Sq, a.H, a.B), dim3(HD), 0, s, a, kv);
  } else {
    hipLaunchKernelGGL((attn_kernel<T, HD, false, false>), dim3(cdiv(a.Sq, kQT), a.H, a.B), dim3(kThreads), 0, s, a,
                       scale, 1);
  }
  return hipGetLastError();
}

}  // namespace

size_t attn_partial_bytes(int B, int H, int Sq, int hd) {
  // the split layout with few workgroups; at most kKvMaxSplits key ranges
  const bool split = Sq <= kSplitMaxQ || cdiv(Sq, kQT) * H * B < kSplitMaxWg;
  if (!split || cdiv(Sq, kQW) * H * B >= kKvMinWg) return 0;
  return size_t(kKvMaxSplits) * B * H * Sq * kv_rec(hd) * sizeof(float);
}

hipError_t attention(int dtype, const AttnArgs& a, hipStream_t s) {
  if (dtype) return a.hd == 128 ? launch_attn<bf16_t, 128>(a, s) : launch_attn<bf16_t, 64>(a, s);
  return a.hd == 128 ? launch_attn<float, 128>(a, s) : launch_attn<float, 64>(a, s);
}

}  // namespace dllm
