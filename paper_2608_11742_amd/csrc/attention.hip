// Full non-causal softmax attention, softmax(q k^T / sqrt(hd)) v over every
// key of the sequence, optionally preceded by the keys of a cached prefix
// (shared by all sequences of the batch).
//
// A workgroup of 4 waves takes 128 queries of one (sequence, head); each
// wave owns 32 queries.  Keys stream through LDS in tiles of 64 (K rows and
// V^T columns, double-buffered, next tile prefetched into registers).
// Scores are computed transposed, S^T = K Q^T, so in the MFMA output layout
// every lane holds one query's scores for 4 keys per 16-key block: the
// online-softmax max/sum and the output rescale stay per lane, and the
// probabilities feed the P V product (computed as O^T = V^T P^T) directly as
// MFMA operands without an LDS round trip.
#include "kernels.h"
#include "common.h"

namespace dllm {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * kWave;
constexpr int kQW = 32;             // queries per wave
constexpr int kQT = kWaves * kQW;   // queries per workgroup
constexpr int kKT = 64;             // keys per tile

template <typename T, int HD>
struct AttnCfg {
  static constexpr int E = Elem<T>::per_chunk;             // elements per 16-byte chunk
  static constexpr int CK = HD * Elem<T>::bytes / 16;      // chunks per K row
  static constexpr int CV = kKT * Elem<T>::bytes / 16;     // chunks per V^T row (64 keys)
  static constexpr int KB = kKT * CK * 16;                 // K tile bytes
  static constexpr int VB = HD * CV * 16;                  // V^T tile bytes
  static constexpr int STAGE = KB + VB;
  static constexpr int KLD = kKT * CK / kThreads;          // K chunks per thread
  static constexpr int VLD = HD * CV / kThreads;           // V chunks per thread
  static constexpr int NDB = HD / 16;                      // 16-row dim blocks of O^T
  static constexpr int QSTEPS = CK / 4;                    // MFMA k-steps over head_dim
  static_assert(KLD * kThreads == kKT * CK && VLD * kThreads == HD * CV, "tile split");
};

__device__ __forceinline__ int swz(int r, int c, int row_bytes) { return r * row_bytes + ((c ^ (r & 7)) << 4); }

template <typename T, int HD>
__global__ __launch_bounds__(kThreads, (HD * Elem<T>::bytes >= 256 ? 1 : 2)) void attn_kernel(AttnArgs a,
                                                                                              float qk_scale_log2) {
  using C = AttnCfg<T, HD>;
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * C::STAGE];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int fr = lane & 15, g = lane >> 4;
  const int b = blockIdx.z, h = blockIdx.y;
  const int q0 = blockIdx.x * kQT + wave * kQW;
  const size_t bh = size_t(b) * a.H + h;

  const T* Q = static_cast<const T*>(a.q) + bh * a.Sq * HD;
  const T* Ko = static_cast<const T*>(a.k) + bh * a.Sq * HD;
  const T* Vo = static_cast<const T*>(a.vt) + bh * HD * a.vt_ld;
  const T* Kp = a.kp ? static_cast<const T*>(a.kp) + size_t(h) * a.p_cap * HD : nullptr;
  const T* Vp = a.kp ? static_cast<const T*>(a.vpt) + size_t(h) * HD * a.p_cap : nullptr;
  const int n_pt = a.kp ? cdiv(a.p_len, kKT) : 0;
  const int n_ot = cdiv(a.Sq, kKT);
  const int n_tiles = n_pt + n_ot;

  // Q fragments (B operand of S^T = K Q^T): query q0 + 16 qb + fr, chunk 4 step + g
  u32x4 qf[2][C::QSTEPS];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int q = min(q0 + qb * 16 + fr, a.Sq - 1);
#pragma unroll
    for (int st = 0; st < C::QSTEPS; ++st)
      qf[qb][st] = *reinterpret_cast<const u32x4*>(reinterpret_cast<const uint8_t*>(Q + size_t(q) * HD) +
                                                   (4 * st + g) * 16);
  }

  // global -> register prefetch of one key tile, K and V^T halves separately
  // (the K half is live during QK^T, the V half during PV)
  u32x4 rk[C::KLD], rv[C::VLD];
  auto gload_k = [&](int t) {
    const bool pre = t < n_pt;
    const int k0 = (pre ? t : t - n_pt) * kKT;
    const int nk = pre ? a.p_len : a.Sq;
    const T* Kb = pre ? Kp : Ko;
#pragma unroll
    for (int i = 0; i < C::KLD; ++i) {
      const int qd = tid + kThreads * i, r = qd / C::CK, c = qd % C::CK;
      const int key = min(k0 + r, nk - 1);
      rk[i] = *reinterpret_cast<const u32x4*>(reinterpret_cast<const uint8_t*>(Kb + size_t(key) * HD) + c * 16);
    }
  };
  auto gload_v = [&](int t) {
    const bool pre = t < n_pt;
    const int k0 = (pre ? t : t - n_pt) * kKT;
    const int nk = pre ? a.p_len : a.Sq;
    const T* Vb = pre ? Vp : Vo;
    const int ld = pre ? a.p_cap : a.vt_ld;
#pragma unroll
    for (int i = 0; i < C::VLD; ++i) {
      const int qd = tid + kThreads * i, r = qd / C::CV, c = qd % C::CV;
      const int key0 = k0 + c * C::E;
      u32x4 v = u32x4{0u, 0u, 0u, 0u};
      if (key0 < nk) {
        v = *reinterpret_cast<const u32x4*>(Vb + size_t(r) * ld + key0);
        if (key0 + C::E > nk) {   // ragged tail: zero the values of keys >= nk
          const int valid = nk - key0;
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const int e_lo = w * (C::E / 4);
            if constexpr (C::E == 8) {
              uint32_t m = (e_lo < valid ? 0xffffu : 0u) | (e_lo + 1 < valid ? 0xffff0000u : 0u);
              v[w] &= m;
            } else {
              if (e_lo >= valid) v[w] = 0u;
            }
          }
        }
      }
      rv[i] = v;
    }
  };
  auto sstore_k = [&](int buf) {
    uint8_t* s = smem + buf * C::STAGE;
#pragma unroll
    for (int i = 0; i < C::KLD; ++i) {
      const int qd = tid + kThreads * i, r = qd / C::CK, c = qd % C::CK;
      *reinterpret_cast<u32x4*>(s + swz(r, c, C::CK * 16)) = rk[i];
    }
  };
  auto sstore_v = [&](int buf) {
    uint8_t* s = smem + buf * C::STAGE;
#pragma unroll
    for (int i = 0; i < C::VLD; ++i) {
      const int qd = tid + kThreads * i, r = qd / C::CV, c = qd % C::CV;
      *reinterpret_cast<u32x4*>(s + C::KB + swz(r, c, C::CV * 16)) = rv[i];
    }
  };

  f32x4 o[C::NDB][2];
#pragma unroll
  for (int db = 0; db < C::NDB; ++db) o[db][0] = o[db][1] = f32x4{0.f, 0.f, 0.f, 0.f};
  float mrun[2] = {-INFINITY, -INFINITY};
  float lrun[2] = {0.f, 0.f};

  gload_k(0);
  gload_v(0);
  sstore_k(0);
  sstore_v(0);
  __syncthreads();
  for (int t = 0; t < n_tiles; ++t) {
    const bool more = t + 1 < n_tiles;
    if (more) gload_k(t + 1);
    const uint8_t* s = smem + (t & 1) * C::STAGE;
    const bool pre = t < n_pt;
    const int nk = pre ? a.p_len : a.Sq;
    const int k0 = (pre ? t : t - n_pt) * kKT;

    const uint8_t* sv = s + C::KB;
    // the tile's 64 keys in two halves of 32: S^T, online softmax and P V per half
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      // S^T block (key block 2 half + kk, query block qb)
      f32x4 sc[2][2];
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const int kb = 2 * half + kk;
        sc[kk][0] = sc[kk][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int st = 0; st < C::QSTEPS; ++st) {
          const u32x4 kf = *reinterpret_cast<const u32x4*>(s + swz(kb * 16 + fr, 4 * st + g, C::CK * 16));
          Mfma<T>::run(sc[kk][0], kf, qf[0][st]);
          Mfma<T>::run(sc[kk][1], kf, qf[1][st]);
        }
      }
      if (half == 1 && more) {
        sstore_k((t + 1) & 1);   // the other buffer's K half was last read before the previous barrier
        gload_v(t + 1);
      }
      // online softmax per query column (this lane's query q0 + 16 qb + fr)
      float p[2][2][4];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
        float mt = -INFINITY;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int key = k0 + (2 * half + kk) * 16 + 4 * g + i;
            const float v = key < nk ? sc[kk][qb][i] * qk_scale_log2 : -INFINITY;
            p[kk][qb][i] = v;
            mt = fmaxf(mt, v);
          }
        mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
        mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
        const float mnew = fmaxf(mrun[qb], mt);
        const float alpha = __builtin_amdgcn_exp2f(mrun[qb] - mnew);
        mrun[qb] = mnew;
        float ls = 0.f;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float e = __builtin_amdgcn_exp2f(p[kk][qb][i] - mnew);
            p[kk][qb][i] = e;
            ls += e;
          }
        lrun[qb] = lrun[qb] * alpha + ls;
#pragma unroll
        for (int db = 0; db < C::NDB; ++db) o[db][qb] *= alpha;
      }
      // O^T += V^T P^T over keys 32 half .. 32 half + 31
      if constexpr (Elem<T>::per_chunk == 8) {
        // P enters the product as a pair of bf16 values, hi = bf16(p) and
        // lo = bf16(p - hi), so the weights keep about 16 significant bits.
        u32x4 ph[2], pl[2];
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const int kk = w >> 1, i0 = 2 * (w & 1);
            const float a0 = p[kk][qb][i0], a1 = p[kk][qb][i0 + 1];
            const uint16_t h0 = f2bf(a0), h1 = f2bf(a1);
            ph[qb][w] = uint32_t(h0) | (uint32_t(h1) << 16);
            pl[qb][w] = uint32_t(f2bf(a0 - bf2f(h0))) | (uint32_t(f2bf(a1 - bf2f(h1))) << 16);
          }
#pragma unroll
        for (int db = 0; db < C::NDB; ++db) {
          const int r = db * 16 + fr;
          const int ka = 32 * half + 4 * g, kbk = ka + 16;   // key offsets of the two 4-key halves
          const u32x2 lo = *reinterpret_cast<const u32x2*>(sv + swz(r, ka >> 3, C::CV * 16) + (ka & 7) * 2);
          const u32x2 hi = *reinterpret_cast<const u32x2*>(sv + swz(r, kbk >> 3, C::CV * 16) + (kbk & 7) * 2);
          const u32x4 vf = u32x4{lo[0], lo[1], hi[0], hi[1]};
#pragma unroll
          for (int qb = 0; qb < 2; ++qb) {
            Mfma<T>::run(o[db][qb], vf, ph[qb]);
            Mfma<T>::run(o[db][qb], vf, pl[qb]);
          }
        }
      } else {
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          u32x4 pb[2];
#pragma unroll
          for (int qb = 0; qb < 2; ++qb)
#pragma unroll
            for (int i = 0; i < 4; ++i) pb[qb][i] = __float_as_uint(p[kk][qb][i]);
#pragma unroll
          for (int db = 0; db < C::NDB; ++db) {
            const int r = db * 16 + fr;
            const int key = (2 * half + kk) * 16 + 4 * g;  // 4 fp32 keys = one chunk
            const u32x4 vf = *reinterpret_cast<const u32x4*>(sv + swz(r, key >> 2, C::CV * 16));
            Mfma<T>::run(o[db][0], vf, pb[0]);
            Mfma<T>::run(o[db][1], vf, pb[1]);
          }
        }
      }
    }
    if (more) sstore_v((t + 1) & 1);
    __syncthreads();
  }

  // normalise and store O[b * Sq + q][h * HD + dim]
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    float l = lrun[qb];
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
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

template <typename T, int HD>
hipError_t launch_attn(const AttnArgs& a, hipStream_t s) {
  const float scale = 1.4426950408889634f / sqrtf(float(HD));
  hipLaunchKernelGGL((attn_kernel<T, HD>), dim3(cdiv(a.Sq, kQT), a.H, a.B), dim3(kThreads), 0, s, a, scale);
  return hipGetLastError();
}

}  // namespace

hipError_t attention(int dtype, const AttnArgs& a, hipStream_t s) {
  if (dtype) return a.hd == 128 ? launch_attn<bf16_t, 128>(a, s) : launch_attn<bf16_t, 64>(a, s);
  return a.hd == 128 ? launch_attn<float, 128>(a, s) : launch_attn<float, 64>(a, s);
}

}  // namespace dllm
