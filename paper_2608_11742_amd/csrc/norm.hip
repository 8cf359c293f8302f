// Row-wise kernels of the forward: embedding gather, RMSNorm (optionally
// gathering rows) and the prefix-cache writer.
#include "kernels.h"
#include "common.h"

namespace dllm {

namespace {

constexpr int kRowThreads = 256;

template <typename T>
__global__ __launch_bounds__(kRowThreads) void embed_kernel(const int32_t* __restrict__ tok, const T* __restrict__ emb,
                                                            int d, int vocab, float* __restrict__ x) {
  const int r = blockIdx.x;
  const int t = min(max(tok[r], 0), vocab - 1);
  const T* src = emb + size_t(t) * d;
  float* dst = x + size_t(r) * d;
  for (int c = threadIdx.x; c < d; c += kRowThreads) dst[c] = load_f(src + c);
}

// store 4 consecutive values as one 8-byte (bf16) or 16-byte (fp32) access
__device__ __forceinline__ void store4(bf16_t* p, f32x4 v) {
  const uint32_t lo = uint32_t(f2bf(v.x)) | (uint32_t(f2bf(v.y)) << 16);
  const uint32_t hi = uint32_t(f2bf(v.z)) | (uint32_t(f2bf(v.w)) << 16);
  *reinterpret_cast<u32x2*>(p) = u32x2{lo, hi};
}
__device__ __forceinline__ void store4(float* p, f32x4 v) { *reinterpret_cast<f32x4*>(p) = v; }

constexpr int kNormChunks = 8;   // 16-byte chunks per thread held in registers: d <= 8192
constexpr int kFewRows = 256;    // fewer rows than CUs: resid_rmsnorm takes kWideThreads per row
constexpr int kWideThreads = 1024;

// One workgroup per output row; the row stays in registers between the sum
// of squares (reduced in fp32 over 4 waves) and the scaled store.
template <typename T>
__global__ __launch_bounds__(kRowThreads) void rmsnorm_kernel(const float* __restrict__ x, int d, float eps,
                                                              const int32_t* __restrict__ pos, int n_pos, int seq,
                                                              T* __restrict__ out) {
  __shared__ float part[kRowThreads / kWave];
  const int r = blockIdx.x;
  const int src_row = pos ? (r / n_pos) * seq + min(max(pos[r % n_pos], 0), seq - 1) : r;
  const float* xr = x + size_t(src_row) * d;
  f32x4 v[kNormChunks];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < kNormChunks; ++j) {
    const int c = (threadIdx.x + j * kRowThreads) * 4;
    v[j] = c < d ? *reinterpret_cast<const f32x4*>(xr + c) : f32x4{0.f, 0.f, 0.f, 0.f};
    ss += v[j].x * v[j].x + v[j].y * v[j].y + v[j].z * v[j].z + v[j].w * v[j].w;
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < kRowThreads / kWave; ++w) tot += part[w];
  const float inv = 1.0f / sqrtf(tot / float(d) + eps);
  T* o = out + size_t(r) * d;
#pragma unroll
  for (int j = 0; j < kNormChunks; ++j) {
    const int c = (threadIdx.x + j * kRowThreads) * 4;
    if (c < d) store4(o + c, v[j] * inv);
  }
}

// Residual update from split-K partial tiles fused with the RMSNorm that
// follows it: x[r] += part[0][r] + part[1][r] + ... (in this order, as the
// separate reduction), then out[r] = x[r] / sqrt(mean(x[r]^2) + eps).
template <typename T, int THREADS>
__global__ __launch_bounds__(THREADS) void resid_rmsnorm_kernel(const float* __restrict__ part, int splits, int np,
                                                                int M, float* __restrict__ x, int d, float eps,
                                                                T* __restrict__ out) {
  constexpr int CH = kNormChunks * kRowThreads / THREADS;   // 16-byte chunks per thread: d <= 8192
  constexpr int LIF = CH <= 2 ? 8 : 4;                       // partial loads in flight per chunk
  __shared__ float red[THREADS / kWave];
  const int r = blockIdx.x;
  float* xr = x + size_t(r) * d;
  auto pr = [&](int p, int c) { return *reinterpret_cast<const f32x4*>(part + (size_t(p) * M + r) * np + c); };
  f32x4 v[CH];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < CH; ++j) {
    const int c = (threadIdx.x + j * THREADS) * 4;
    v[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (c < d) {
      v[j] = *reinterpret_cast<const f32x4*>(xr + c);
      int p = 0;
      for (; p + LIF <= splits; p += LIF) {   // LIF loads in flight, added in order
        f32x4 a[LIF];
#pragma unroll
        for (int q = 0; q < LIF; ++q) a[q] = pr(p + q, c);
#pragma unroll
        for (int q = 0; q < LIF; ++q) v[j] += a[q];
      }
      for (; p < splits; ++p) v[j] += pr(p, c);
      *reinterpret_cast<f32x4*>(xr + c) = v[j];
    }
    ss += v[j].x * v[j].x + v[j].y * v[j].y + v[j].z * v[j].z + v[j].w * v[j].w;
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < THREADS / kWave; ++w) tot += red[w];
  const float inv = 1.0f / sqrtf(tot / float(d) + eps);
  T* o = out + size_t(r) * d;
#pragma unroll
  for (int j = 0; j < CH; ++j) {
    const int c = (threadIdx.x + j * THREADS) * 4;
    if (c < d) store4(o + c, v[j] * inv);
  }
}

// grid: (H, rows of this call); copies K rows and V^T columns into the cache
template <typename T>
__global__ __launch_bounds__(kRowThreads) void kv_store_kernel(const T* __restrict__ k, const T* __restrict__ vt,
                                                               int seq, int hd, int vt_ld, T* __restrict__ ck,
                                                               T* __restrict__ cvt, int cap, int off) {
  const int h = blockIdx.x, s = blockIdx.y;
  for (int c = threadIdx.x; c < hd; c += kRowThreads) {
    ck[(size_t(h) * cap + off + s) * hd + c] = k[(size_t(h) * seq + s) * hd + c];
    cvt[(size_t(h) * hd + c) * cap + off + s] = vt[(size_t(h) * hd + c) * vt_ld + s];
  }
}

}  // namespace

hipError_t embed(int dtype, const int32_t* tok, int rows, const void* emb, int d, int vocab, float* x, hipStream_t s) {
  if (dtype)
    hipLaunchKernelGGL(embed_kernel<bf16_t>, dim3(rows), dim3(kRowThreads), 0, s, tok,
                       static_cast<const bf16_t*>(emb), d, vocab, x);
  else
    hipLaunchKernelGGL(embed_kernel<float>, dim3(rows), dim3(kRowThreads), 0, s, tok,
                       static_cast<const float*>(emb), d, vocab, x);
  return hipGetLastError();
}

hipError_t rmsnorm(int dtype, const float* x, int d, float eps, int rows, const int32_t* pos, int n_pos, int seq,
                   void* out, hipStream_t s) {
  if (d % 4 || d > kNormChunks * kRowThreads * 4) return hipErrorInvalidValue;
  if (dtype)
    hipLaunchKernelGGL(rmsnorm_kernel<bf16_t>, dim3(rows), dim3(kRowThreads), 0, s, x, d, eps, pos, n_pos, seq,
                       static_cast<bf16_t*>(out));
  else
    hipLaunchKernelGGL(rmsnorm_kernel<float>, dim3(rows), dim3(kRowThreads), 0, s, x, d, eps, pos, n_pos, seq,
                       static_cast<float*>(out));
  return hipGetLastError();
}

hipError_t resid_rmsnorm(int dtype, const float* part, int splits, int np, int M, float* x, int d, float eps,
                         void* out, hipStream_t s) {
  if (d % 4 || np % 4 || d > kNormChunks * kRowThreads * 4) return hipErrorInvalidValue;
  // Fewer rows than CUs: 1024 threads per row, so that each thread walks the
  // partials of fewer columns with more loads in flight.
  const bool wide = M < kFewRows;
  if (dtype) {
    if (wide)
      hipLaunchKernelGGL((resid_rmsnorm_kernel<bf16_t, kWideThreads>), dim3(M), dim3(kWideThreads), 0, s, part,
                         splits, np, M, x, d, eps, static_cast<bf16_t*>(out));
    else
      hipLaunchKernelGGL((resid_rmsnorm_kernel<bf16_t, kRowThreads>), dim3(M), dim3(kRowThreads), 0, s, part,
                         splits, np, M, x, d, eps, static_cast<bf16_t*>(out));
  } else {
    if (wide)
      hipLaunchKernelGGL((resid_rmsnorm_kernel<float, kWideThreads>), dim3(M), dim3(kWideThreads), 0, s, part,
                         splits, np, M, x, d, eps, static_cast<float*>(out));
    else
      hipLaunchKernelGGL((resid_rmsnorm_kernel<float, kRowThreads>), dim3(M), dim3(kRowThreads), 0, s, part,
                         splits, np, M, x, d, eps, static_cast<float*>(out));
  }
  return hipGetLastError();
}

hipError_t kv_store(int dtype, const void* k, const void* vt, int H, int seq, int hd, int vt_ld, void* ck,
                    void* cvt, int cap, int off, hipStream_t s) {
  if (dtype)
    hipLaunchKernelGGL(kv_store_kernel<bf16_t>, dim3(H, seq), dim3(kRowThreads), 0, s,
                       static_cast<const bf16_t*>(k), static_cast<const bf16_t*>(vt), seq, hd, vt_ld,
                       static_cast<bf16_t*>(ck), static_cast<bf16_t*>(cvt), cap, off);
  else
    hipLaunchKernelGGL(kv_store_kernel<float>, dim3(H, seq), dim3(kRowThreads), 0, s,
                       static_cast<const float*>(k), static_cast<const float*>(vt), seq, hd, vt_ld,
                       static_cast<float*>(ck), static_cast<float*>(cvt), cap, off);
  return hipGetLastError();
}

namespace {

// LM-head row t = c * n_lm + j reads position lm_pos[j] of sequence c: the
// shared sequence for c = 0, branch c-1's copy of the block for c >= 1 when
// the position lies in the block (else the shared row)
__global__ void packed_lm_rows_kernel(int S, int b0, int B, int R, const int32_t* __restrict__ lm_pos, int n_lm,
                                      int32_t* __restrict__ row, int32_t* __restrict__ src) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= R) return;
  const int c = t / n_lm;
  const int p = min(max(lm_pos[t - c * n_lm], 0), S - 1);
  row[t] = (c > 0 && p >= b0 && p < b0 + B) ? S + (c - 1) * B + (p - b0) : p;
  src[t] = p;
}

}  // namespace

hipError_t packed_lm_rows(int S, int b0, int B, int n_branch, const int32_t* lm_pos, int n_lm, int32_t* row,
                          int32_t* src, hipStream_t s) {
  const int R = (1 + n_branch) * n_lm;
  hipLaunchKernelGGL(packed_lm_rows_kernel, dim3(cdiv(R, 256)), dim3(256), 0, s, S, b0, B, R, lm_pos, n_lm, row,
                     src);
  return hipGetLastError();
}

}  // namespace dllm
