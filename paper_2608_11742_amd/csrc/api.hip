// Host side of the C ABI: argument validation, workspace planning and the
// stream-ordered launch sequence of one denoising forward and of the
// scheduler calls.  Nothing here allocates except dllm_model_create.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "dllm_rps.h"
#include "kernels.h"

using namespace dllm;

struct dllm_model {
  dllm_model_desc desc;
  const void* emb;
  const void* lm_head;
  std::vector<const void*> wqkv, wo, wgu, wdown;
  float2* rope;
  // kernel timing (dllm_profile_begin / end)
  std::vector<hipEvent_t> prof_ev;   // 2 per launch
  std::vector<int> prof_cls;
  int prof_used = 0;
  bool prof_on = false;
  uint32_t prof_mask = ~0u;   // classes bracketed while profiling
};

namespace {

// Brackets one launch with events when profiling is on.
struct ProfScope {
  dllm_model* m;
  hipStream_t s;
  int idx = -1;
  ProfScope(dllm_model* m_, hipStream_t s_, int cls) : m(m_), s(s_) {
    if (!m->prof_on || !((m->prof_mask >> cls) & 1u) || m->prof_used >= int(m->prof_cls.size())) return;
    idx = m->prof_used++;
    m->prof_cls[idx] = cls;
    (void)hipEventRecord(m->prof_ev[2 * idx], s);
  }
  ~ProfScope() {
    if (idx >= 0) (void)hipEventRecord(m->prof_ev[2 * idx + 1], s);
  }
};

}  // namespace

namespace {

thread_local std::string g_err;

dllm_status fail(dllm_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
dllm_status fail(dllm_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

dllm_status hip_check(hipError_t e, const char* what) {
  if (e == hipSuccess) return DLLM_OK;
  return fail(DLLM_EHIP, "%s: %s", what, hipGetErrorString(e));
}

#define TRY_HIP(expr, what)                         \
  do {                                              \
    dllm_status st_ = hip_check((expr), (what));    \
    if (st_ != DLLM_OK) return st_;                 \
  } while (0)

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
int elem_bytes(int dtype) { return dtype == DLLM_BF16 ? 2 : 4; }

StatsOut to_out(const dllm_stats& s) {
  return StatsOut{s.H, s.lse, s.lmax, s.argmax, s.topk_id, s.topk_logit, s.k};
}

dllm_status check_stats(const dllm_stats* s, const char* name) {
  if (!s) return fail(DLLM_EINVAL, "%s is NULL", name);
  if (!s->H || !s->lse || !s->lmax || !s->argmax || !s->topk_id || !s->topk_logit)
    return fail(DLLM_EINVAL, "%s has a NULL array", name);
  if (s->k < 1 || s->k > DLLM_MAX_TOPK) return fail(DLLM_EINVAL, "%s.k = %d outside 1..%d", name, s->k, DLLM_MAX_TOPK);
  return DLLM_OK;
}

// Workspace layout of one forward (256-byte aligned regions).
struct FwdLayout {
  size_t x, a, q, k, vt, f, hl, lm, lmsrc, part, attn, total;
  int vt_ld;
};

// split-K parts of the four projections of a forward over M rows, and the
// partial-tile workspace they share (one projection at a time)
struct GemmSplits {
  int qkv, o, gu, down;
  size_t bytes;
};

GemmSplits plan_gemms(const dllm_model_desc& d, int M) {
  const int dt = d.dtype;
  auto cdiv = [](int a, int b) { return (a + b - 1) / b; };
  const int tq = cdiv(3 * d.d_model, 256), to = cdiv(d.d_model, 256), tg = cdiv(d.d_ffn, 128);
  GemmSplits g;
  g.qkv = gemm_splits(GEMM_KIND_QKV, M, 3 * d.d_model, d.d_model, dt);
  g.o = gemm_splits(GEMM_KIND_RESID, M, d.d_model, d.d_model, dt);
  g.gu = d.d_ffn % 4 ? 1 : gemm_splits(GEMM_KIND_GATEUP, M, 2 * d.d_ffn, d.d_model, dt);
  g.down = gemm_splits(GEMM_KIND_RESID, M, d.d_model, d.d_ffn, dt);
  g.bytes = std::max(std::max(gemm_partial_bytes(M, tq, g.qkv), gemm_partial_bytes(M, to, g.o)),
                     std::max(gemm_partial_bytes(M, tg, g.gu), gemm_partial_bytes(M, to, g.down)));
  return g;
}

// packed lookahead layout of one forward (see dllm_forward_packed)
struct Packing {
  int S, b0, B, n_branch;
};

// R: LM-head rows of the call (batch * n_lm_pos, or (1 + n_branch) * n_lm_pos packed)
FwdLayout plan_forward(const dllm_model_desc& d, int batch, int seq, int R) {
  FwdLayout L;
  const size_t T = elem_bytes(d.dtype);
  const size_t M = size_t(batch) * seq;
  L.vt_ld = int(align_up(seq, 8));
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes, 256);
    return o;
  };
  L.x = take(M * d.d_model * 4);
  L.a = take(M * d.d_model * T);
  L.q = take(M * d.d_model * T);
  L.k = take(M * d.d_model * T);
  L.vt = take(size_t(batch) * d.n_heads * d.head_dim * L.vt_ld * T);
  L.f = take(M * d.d_ffn * T);
  L.hl = take(size_t(R) * d.d_model * T);
  L.lm = take(lmhead_workspace(R, d.vocab));
  L.lmsrc = take(size_t(R) * 8);
  L.part = take(plan_gemms(d, int(M)).bytes);
  const size_t attn_bytes = attn_partial_bytes(batch, d.n_heads, seq, d.head_dim);
  L.attn = attn_bytes ? take(attn_bytes) : 0;
  L.total = off;
  return L;
}

}  // namespace

extern "C" {

int32_t dllm_abi_version(void) { return DLLM_ABI_VERSION; }

const char* dllm_last_error(void) { return g_err.c_str(); }

const char* dllm_status_string(dllm_status s) {
  switch (s) {
    case DLLM_OK: return "ok";
    case DLLM_EINVAL: return "invalid argument";
    case DLLM_ESHAPE: return "unsupported shape";
    case DLLM_EDTYPE: return "unknown dtype";
    case DLLM_ENOMEM: return "workspace too small";
    case DLLM_EHIP: return "HIP runtime error";
    case DLLM_EUNSUPPORTED: return "unsupported";
  }
  return "unknown status";
}

dllm_status dllm_model_create(const dllm_model_desc* desc, const dllm_weights* w, dllm_model** out) {
  if (!desc || !w || !out) return fail(DLLM_EINVAL, "dllm_model_create: NULL argument");
  *out = nullptr;
  const dllm_model_desc& d = *desc;
  if (d.dtype != DLLM_F32 && d.dtype != DLLM_BF16) return fail(DLLM_EDTYPE, "dtype %d", d.dtype);
  if (d.n_layers < 1 || d.n_heads < 1 || d.vocab < 2 || d.d_ffn < 1 || d.max_pos < 1)
    return fail(DLLM_ESHAPE, "non-positive model size");
  if (d.head_dim != 64 && d.head_dim != 128) return fail(DLLM_ESHAPE, "head_dim %d not in {64, 128}", d.head_dim);
  if (d.d_model != d.n_heads * d.head_dim) return fail(DLLM_ESHAPE, "d_model != n_heads * head_dim");
  if (d.d_model % 256 || d.d_model > 8192) return fail(DLLM_ESHAPE, "d_model %% 256 != 0 or d_model > 8192");
  if (d.d_ffn % 128) return fail(DLLM_ESHAPE, "d_ffn %% 128 != 0");
  if (d.mask_id < 0 || d.mask_id >= d.vocab) return fail(DLLM_EINVAL, "mask_id outside [0, vocab)");
  if (!(d.rms_eps > 0.f) || !(d.rope_base > 1.f)) return fail(DLLM_EINVAL, "rms_eps / rope_base");
  const size_t T = elem_bytes(d.dtype);
  if (size_t(d.vocab) * d.d_model * T >= (size_t(1) << 32) || size_t(2) * d.d_ffn * d.d_model * T >= (size_t(1) << 32))
    return fail(DLLM_ESHAPE, "a weight matrix exceeds 4 GiB");
  if (!w->emb || !w->lm_head || !w->wqkv || !w->wo || !w->wgu || !w->wdown)
    return fail(DLLM_EINVAL, "NULL weight pointer");
  for (int l = 0; l < d.n_layers; ++l)
    if (!w->wqkv[l] || !w->wo[l] || !w->wgu[l] || !w->wdown[l]) return fail(DLLM_EINVAL, "NULL weight of layer %d", l);

  // rotary table in double precision: angle = pos * base^(-2j/hd)
  const int half = d.head_dim / 2;
  std::vector<float2> tab(size_t(d.max_pos) * half);
  for (int p = 0; p < d.max_pos; ++p)
    for (int j = 0; j < half; ++j) {
      const double ang = double(p) * std::pow(double(d.rope_base), -2.0 * j / d.head_dim);
      tab[size_t(p) * half + j] = make_float2(float(std::cos(ang)), float(std::sin(ang)));
    }
  float2* rope = nullptr;
  TRY_HIP(hipMalloc(&rope, tab.size() * sizeof(float2)), "hipMalloc(rope table)");
  hipError_t e = hipMemcpy(rope, tab.data(), tab.size() * sizeof(float2), hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(rope);
    return hip_check(e, "hipMemcpy(rope table)");
  }
  dllm_model* m = new dllm_model;
  m->desc = d;
  m->emb = w->emb;
  m->lm_head = w->lm_head;
  m->wqkv.assign(w->wqkv, w->wqkv + d.n_layers);
  m->wo.assign(w->wo, w->wo + d.n_layers);
  m->wgu.assign(w->wgu, w->wgu + d.n_layers);
  m->wdown.assign(w->wdown, w->wdown + d.n_layers);
  m->rope = rope;
  *out = m;
  return DLLM_OK;
}

void dllm_model_destroy(dllm_model* m) {
  if (!m) return;
  for (hipEvent_t e : m->prof_ev) (void)hipEventDestroy(e);
  (void)hipFree(m->rope);
  delete m;
}

dllm_status dllm_profile_begin(dllm_model* m, int32_t max_launches) {
  return dllm_profile_begin_classes(m, max_launches, ~0u);
}

dllm_status dllm_profile_begin_classes(dllm_model* m, int32_t max_launches, uint32_t class_mask) {
  if (!m || max_launches < 1) return fail(DLLM_EINVAL, "dllm_profile_begin: NULL model or max_launches < 1");
  if (class_mask == 0) return fail(DLLM_EINVAL, "dllm_profile_begin_classes: empty class mask");
  m->prof_mask = class_mask;
  const size_t need = size_t(2) * max_launches;
  while (m->prof_ev.size() < need) {
    hipEvent_t e;
    TRY_HIP(hipEventCreate(&e), "hipEventCreate");
    m->prof_ev.push_back(e);
  }
  m->prof_cls.assign(max_launches, 0);
  m->prof_used = 0;
  m->prof_on = true;
  return DLLM_OK;
}

dllm_status dllm_profile_end(dllm_model* m, float* ms, int32_t* launches) {
  if (!m || !ms || !launches) return fail(DLLM_EINVAL, "dllm_profile_end: NULL argument");
  if (!m->prof_on) return fail(DLLM_EINVAL, "dllm_profile_end without dllm_profile_begin");
  m->prof_on = false;
  for (int c = 0; c < DLLM_PROF_CLASSES; ++c) {
    ms[c] = 0.f;
    launches[c] = 0;
  }
  for (int i = 0; i < m->prof_used; ++i) {
    TRY_HIP(hipEventSynchronize(m->prof_ev[2 * i + 1]), "hipEventSynchronize");
    float t = 0.f;
    TRY_HIP(hipEventElapsedTime(&t, m->prof_ev[2 * i], m->prof_ev[2 * i + 1]), "hipEventElapsedTime");
    ms[m->prof_cls[i]] += t;
    launches[m->prof_cls[i]] += 1;
  }
  m->prof_used = 0;
  return DLLM_OK;
}

dllm_status dllm_mfma_ceiling(int32_t random_operands, float* tflops, dllm_stream stream) {
  if (!tflops) return fail(DLLM_EINVAL, "dllm_mfma_ceiling: NULL tflops");
  hipStream_t s = static_cast<hipStream_t>(stream);
  int dev = 0, cus = 0;
  TRY_HIP(hipGetDevice(&dev), "hipGetDevice");
  TRY_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev), "hipDeviceGetAttribute");
  const int wg = 2 * std::max(cus, 1);
  double flop = 0.0;
  TRY_HIP(dllm::mfma_calibration(random_operands != 0, 2000, wg, &flop, s), "mfma_calibration (warm-up)");
  hipEvent_t e0, e1;
  TRY_HIP(hipEventCreate(&e0), "hipEventCreate");
  if (hipEventCreate(&e1) != hipSuccess) {
    (void)hipEventDestroy(e0);
    return fail(DLLM_EHIP, "hipEventCreate");
  }
  float ms = 0.f;
  hipError_t e = hipEventRecord(e0, s);
  if (e == hipSuccess) e = dllm::mfma_calibration(random_operands != 0, 20000, wg, &flop, s);
  if (e == hipSuccess) e = hipEventRecord(e1, s);
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  TRY_HIP(e, "mfma_calibration");
  *tflops = ms > 0.f ? float(flop / (double(ms) * 1e-3) / 1e12) : 0.f;
  return DLLM_OK;
}

size_t dllm_workspace_bytes(const dllm_model* m, int32_t batch, int32_t seq, int32_t n_lm_pos) {
  if (!m || batch < 1 || seq < 1 || n_lm_pos < 1) return 0;
  return plan_forward(m->desc, batch, seq, batch * n_lm_pos).total;
}

size_t dllm_workspace_bytes_packed(const dllm_model* m, int32_t shared_len, int32_t block_len, int32_t n_branch,
                                   int32_t n_lm_pos) {
  if (!m || shared_len < 1 || block_len < 1 || n_branch < 0 || n_lm_pos < 1) return 0;
  return plan_forward(m->desc, 1, shared_len + n_branch * block_len, (1 + n_branch) * n_lm_pos).total;
}

namespace {

dllm_status forward_impl(dllm_model* m, const int32_t* tokens, int32_t batch, int32_t seq, int32_t pos_offset,
                         const dllm_kv_cache* kv_prefix, const dllm_kv_cache* kv_out, const int32_t* lm_pos,
                         int32_t n_lm_pos, const float* row_scale, float scale, const dllm_probe* probe,
                         const dllm_stats* out, void* ws, size_t ws_bytes, dllm_stream stream, const Packing* pk) {
  if (!m) return fail(DLLM_EINVAL, "dllm_forward: NULL model");
  if (!tokens || !lm_pos || !ws) return fail(DLLM_EINVAL, "dllm_forward: NULL tokens, lm_pos or ws");
  dllm_status st = check_stats(out, "out");
  if (st != DLLM_OK) return st;
  const dllm_model_desc& d = m->desc;
  if (batch < 1 || seq < 1 || n_lm_pos < 1 || n_lm_pos > (pk ? pk->S : seq))
    return fail(DLLM_ESHAPE, "batch %d seq %d n_lm_pos %d", batch, seq, n_lm_pos);
  const int n_pos = pk ? pk->S : seq;   // distinct positions of the call
  if (pos_offset < 0 || pos_offset + n_pos > d.max_pos)
    return fail(DLLM_ESHAPE, "positions %d..%d exceed max_pos %d", pos_offset, pos_offset + n_pos - 1, d.max_pos);
  if (pk) {
    if (batch != 1 || kv_out) return fail(DLLM_EINVAL, "packed lookahead: batch 1, no kv_out");
    if (pk->S < 1 || pk->B < 1 || (pk->B & (pk->B - 1)) || pk->n_branch < 0 || seq != pk->S + pk->n_branch * pk->B ||
        pk->b0 < 0 || pk->b0 + pk->B > pk->S)
      return fail(DLLM_ESHAPE, "packed lookahead: shared %d block %d..%d, seq %d", pk->S, pk->b0, pk->b0 + pk->B - 1,
                  seq);
  }
  if (!std::isfinite(scale)) return fail(DLLM_EINVAL, "scale is not finite");
  const size_t T = elem_bytes(d.dtype);
  const size_t M = size_t(batch) * seq;
  if (M * std::max(d.d_model, d.d_ffn) * T >= (size_t(1) << 32) || M > (size_t(1) << 24))
    return fail(DLLM_ESHAPE, "batch * seq too large");
  if (kv_prefix) {
    if (!kv_prefix->k || !kv_prefix->vt) return fail(DLLM_EINVAL, "kv_prefix has a NULL array");
    if (kv_prefix->len < 1 || kv_prefix->len > kv_prefix->cap || kv_prefix->cap % 8)
      return fail(DLLM_ESHAPE, "kv_prefix len %d cap %d (need 1 <= len <= cap, cap %% 8 == 0)", kv_prefix->len,
                  kv_prefix->cap);
  }
  if (kv_out) {
    if (!kv_out->k || !kv_out->vt) return fail(DLLM_EINVAL, "kv_out has a NULL array");
    if (batch != 1) return fail(DLLM_ESHAPE, "kv_out needs batch == 1");
    if (pos_offset + seq > kv_out->cap || kv_out->cap % 8) return fail(DLLM_ESHAPE, "kv_out capacity");
  }
  if (probe && probe->n > 0 && (!probe->row || !probe->token || !probe->logit))
    return fail(DLLM_EINVAL, "probe has a NULL array");
  // LM-head rows: every sequence's n_lm_pos rows; packed: the anchor's, then each branch's
  const int R = (pk ? 1 + pk->n_branch : batch) * n_lm_pos;
  const FwdLayout L = plan_forward(d, batch, seq, R);
  if (ws_bytes < L.total) return fail(DLLM_ENOMEM, "workspace %zu < %zu bytes", ws_bytes, L.total);

  hipStream_t s = static_cast<hipStream_t>(stream);
  uint8_t* base = static_cast<uint8_t*>(ws);
  float* x = reinterpret_cast<float*>(base + L.x);
  void* a = base + L.a;
  void* q = base + L.q;
  void* k = base + L.k;
  void* vt = base + L.vt;
  void* f = base + L.f;
  void* hl = base + L.hl;
  const int dm = d.d_model, F = d.d_ffn, H = d.n_heads, hd = d.head_dim, dt = d.dtype;
  const int Mi = int(M);
  const GemmSplits gs = plan_gemms(d, Mi);
  float* part = reinterpret_cast<float*>(base + L.part);
  // the residual projections leave their partials to the RMSNorm that follows
  const SplitK sk_qkv{part, gs.qkv}, sk_o{part, gs.o, true}, sk_gu{part, gs.gu}, sk_down{part, gs.down, true};
  const int np_d = (dm + 255) / 256 * 256;   // partial row pitch of the d-wide projections
  int pending = 0;                            // split-K parts of x not yet added (0: none)
  // gathered row of each LM-head row (indexed modulo lm_n, per sequence) and
  // its row-scale index (its in-sequence position)
  const int32_t* lm_row = lm_pos;
  const int32_t* rs_idx = lm_pos;
  int lm_n = n_lm_pos;
  if (pk) {
    int32_t* rows = reinterpret_cast<int32_t*>(base + L.lmsrc);
    ProfScope ps(m, s, DLLM_PROF_OTHER);
    TRY_HIP(packed_lm_rows(pk->S, pk->b0, pk->B, pk->n_branch, lm_pos, n_lm_pos, rows, rows + R, s),
            "packed LM-head rows");
    lm_row = rows;
    rs_idx = rows + R;
    lm_n = R;
  }

  {
    ProfScope ps(m, s, DLLM_PROF_EMBED);
    TRY_HIP(embed(dt, tokens, Mi, m->emb, dm, d.vocab, x, s), "embed");
  }
  // a = rmsnorm(x), first adding the pending split-K partials of the last residual projection
  auto norm_into_a = [&]() -> dllm_status {
    ProfScope ps(m, s, DLLM_PROF_RMSNORM);
    if (pending > 1)
      TRY_HIP(resid_rmsnorm(dt, part, pending, np_d, Mi, x, dm, d.rms_eps, a, s), "resid_rmsnorm");
    else
      TRY_HIP(rmsnorm(dt, x, dm, d.rms_eps, Mi, nullptr, 1, seq, a, s), "rmsnorm");
    pending = 0;
    return DLLM_OK;
  };
  for (int l = 0; l < d.n_layers; ++l) {
    if (dllm_status e = norm_into_a(); e != DLLM_OK) return e;
    QkvOut qo{q, k, vt, seq, L.vt_ld, pos_offset, H, hd, dm, m->rope};
    if (pk) {
      qo.pack_S = pk->S;
      qo.pack_b0 = pk->b0;
      qo.pack_B = pk->B;
    }
    {
      ProfScope ps(m, s, DLLM_PROF_GEMM_QKV);
      TRY_HIP(gemm_qkv(dt, a, dm, m->wqkv[l], Mi, dm, qo, s, &sk_qkv), "gemm_qkv");
    }
    if (kv_out) {
      const size_t lay = size_t(l) * H * kv_out->cap * hd * T;
      ProfScope ps(m, s, DLLM_PROF_OTHER);
      TRY_HIP(kv_store(dt, k, vt, H, seq, hd, L.vt_ld, static_cast<uint8_t*>(kv_out->k) + lay,
                       static_cast<uint8_t*>(kv_out->vt) + lay, kv_out->cap, pos_offset, s),
              "kv_store");
    }
    AttnArgs aa{};
    aa.q = q;
    aa.k = k;
    aa.vt = vt;
    aa.B = batch;
    aa.H = H;
    aa.Sq = seq;
    aa.hd = hd;
    aa.vt_ld = L.vt_ld;
    if (kv_prefix) {
      const size_t lay = size_t(l) * H * kv_prefix->cap * hd * T;
      aa.kp = static_cast<const uint8_t*>(kv_prefix->k) + lay;
      aa.vpt = static_cast<const uint8_t*>(kv_prefix->vt) + lay;
      aa.p_len = kv_prefix->len;
      aa.p_cap = kv_prefix->cap;
    }
    aa.o = a;
    if (L.attn) aa.kv_part = reinterpret_cast<float*>(base + L.attn);
    if (pk) {
      aa.pack_S = pk->S;
      aa.pack_b0 = pk->b0;
      aa.pack_B = pk->B;
    }
    {
      ProfScope ps(m, s, DLLM_PROF_ATTENTION);
      TRY_HIP(attention(dt, aa, s), "attention");
    }
    {
      ProfScope ps(m, s, DLLM_PROF_GEMM_O);
      TRY_HIP(gemm_resid(dt, a, dm, m->wo[l], dm, Mi, dm, dm, x, dm, s, &sk_o), "gemm_o");
      pending = sk_o.splits;
    }
    if (dllm_status e = norm_into_a(); e != DLLM_OK) return e;
    {
      ProfScope ps(m, s, DLLM_PROF_GEMM_GATEUP);
      TRY_HIP(gemm_swiglu(dt, a, dm, m->wgu[l], Mi, F, dm, f, s, &sk_gu), "gemm_swiglu");
    }
    {
      ProfScope ps(m, s, DLLM_PROF_GEMM_DOWN);
      TRY_HIP(gemm_resid(dt, f, F, m->wdown[l], F, Mi, dm, F, x, dm, s, &sk_down), "gemm_down");
      pending = sk_down.splits;
    }
  }
  if (pending > 1) {
    ProfScope ps(m, s, DLLM_PROF_GEMM_DOWN);
    TRY_HIP(splitk_add(sk_down, Mi, dm, x, dm, s), "split-K residual");
  }
  {
    ProfScope ps(m, s, DLLM_PROF_RMSNORM);
    TRY_HIP(rmsnorm(dt, x, dm, d.rms_eps, R, lm_row, lm_n, seq, hl, s), "final rmsnorm");
  }
  {
    ProfScope ps(m, s, DLLM_PROF_LMHEAD);
    TRY_HIP(lmhead_partials(dt, hl, m->lm_head, R, dm, d.vocab, row_scale, rs_idx, lm_n, n_pos, scale,
                            d.mask_id, base + L.lm, s),
            "lm head");
  }
  {
    ProfScope ps(m, s, DLLM_PROF_LMHEAD_MERGE);
    TRY_HIP(lmhead_merge(R, d.vocab, to_out(*out), base + L.lm, s), "lm head merge");
  }
  if (probe && probe->n > 0) {
    ProfScope ps(m, s, DLLM_PROF_OTHER);
    TRY_HIP(probe_logits(dt, hl, m->lm_head, dm, d.vocab, R, probe->row, probe->token, probe->n, row_scale, rs_idx,
                         lm_n, n_pos, scale, probe->logit, s),
            "probe");
  }
  return DLLM_OK;
}

}  // namespace

dllm_status dllm_forward(dllm_model* m, const int32_t* tokens, int32_t batch, int32_t seq, int32_t pos_offset,
                         const dllm_kv_cache* kv_prefix, const dllm_kv_cache* kv_out, const int32_t* lm_pos,
                         int32_t n_lm_pos, const float* row_scale, float scale, const dllm_probe* probe,
                         const dllm_stats* out, void* ws, size_t ws_bytes, dllm_stream stream) {
  return forward_impl(m, tokens, batch, seq, pos_offset, kv_prefix, kv_out, lm_pos, n_lm_pos, row_scale, scale, probe,
                      out, ws, ws_bytes, stream, nullptr);
}

dllm_status dllm_forward_packed(dllm_model* m, const int32_t* tokens, int32_t shared_len, int32_t block_start,
                                int32_t block_len, int32_t n_branch, int32_t pos_offset, const dllm_kv_cache* kv_prefix,
                                const int32_t* lm_pos, int32_t n_lm_pos, const float* row_scale, float scale,
                                const dllm_probe* probe, const dllm_stats* out, void* ws, size_t ws_bytes,
                                dllm_stream stream) {
  if (n_branch < 0 || block_len < 1 || shared_len < 1)
    return fail(DLLM_ESHAPE, "packed lookahead: shared %d, %d branches of %d", shared_len, n_branch, block_len);
  const Packing pk{shared_len, block_start, block_len, n_branch};
  return forward_impl(m, tokens, 1, shared_len + n_branch * block_len, pos_offset, kv_prefix, nullptr, lm_pos,
                      n_lm_pos, row_scale, scale, probe, out, ws, ws_bytes, stream, &pk);
}

size_t vocab_entropy_topk_workspace_bytes(int32_t R, int32_t vocab) {
  if (R < 1 || vocab < 2) return 0;
  return lmhead_workspace(R, vocab);
}

dllm_status vocab_entropy_topk(const void* hidden, const void* w_lm, int32_t R, int32_t d, int32_t vocab,
                               int32_t dtype, const float* row_scale, float scale, int32_t mask_id,
                               const dllm_stats* out, void* ws, size_t ws_bytes, dllm_stream stream) {
  if (!hidden || !w_lm || !ws) return fail(DLLM_EINVAL, "vocab_entropy_topk: NULL hidden, w_lm or ws");
  if (dtype != DLLM_F32 && dtype != DLLM_BF16) return fail(DLLM_EDTYPE, "dtype %d", dtype);
  dllm_status st = check_stats(out, "out");
  if (st != DLLM_OK) return st;
  if (R < 1 || vocab < 2 || d < 1) return fail(DLLM_ESHAPE, "R %d vocab %d d %d", R, vocab, d);
  const int kstage = dtype == DLLM_BF16 ? 64 : 32;
  if (d % kstage) return fail(DLLM_ESHAPE, "d %% %d != 0", kstage);
  const size_t T = elem_bytes(dtype);
  if (size_t(vocab) * d * T >= (size_t(1) << 32) || size_t(R) * d * T >= (size_t(1) << 32))
    return fail(DLLM_ESHAPE, "operand exceeds 4 GiB");
  if (mask_id >= vocab) return fail(DLLM_EINVAL, "mask_id >= vocab");
  if (!std::isfinite(scale)) return fail(DLLM_EINVAL, "scale is not finite");
  const size_t need = lmhead_workspace(R, vocab);
  if (ws_bytes < need) return fail(DLLM_ENOMEM, "workspace %zu < %zu bytes", ws_bytes, need);
  hipStream_t s = static_cast<hipStream_t>(stream);
  TRY_HIP(lmhead_partials(dtype, hidden, w_lm, R, d, vocab, row_scale, nullptr, R, R, scale, mask_id, ws, s),
          "vocab_entropy_topk");
  return hip_check(lmhead_merge(R, vocab, to_out(*out), ws, s), "vocab_entropy_topk merge");
}

// ---------------------------------------------------------------- allocation-free LM head

// Partial statistics of vocab_entropy_topk_noalloc, held by every device the
// library runs on until the process ends.  Host code never passes the array's
// name to a kernel (on the host it is only a stand-in for the symbol): the
// device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) uint8_t scratch[DLLM_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of `scratch` on device `dev`, looked up on the first call
// for that device with the device current.
dllm_status scratch_address(int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices) return fail(DLLM_EUNSUPPORTED, "device %d beyond %d devices", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    int cur = -1;
    TRY_HIP(hipGetDevice(&cur), "hipGetDevice");
    if (cur != dev) TRY_HIP(hipSetDevice(dev), "hipSetDevice");
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) (void)hipSetDevice(cur);
    TRY_HIP(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(DLLM_EHIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return DLLM_OK;
}

}  // namespace

dllm_status vocab_entropy_topk_noalloc(const void* hidden, const void* w_lm, int32_t R, int32_t d, int32_t vocab,
                                       int32_t dtype, const float* row_scale, float scale, int32_t mask_id,
                                       const dllm_stats* out, dllm_stream stream) {
  if (R < 1 || vocab < 2) return fail(DLLM_ESHAPE, "R %d vocab %d", R, vocab);
  const size_t need = lmhead_workspace(R, vocab);
  if (need > size_t(DLLM_NOALLOC_SCRATCH_BYTES))
    return fail(DLLM_ENOMEM, "vocab_entropy_topk_noalloc: R %d x vocab %d needs %zu bytes of partials, beyond the "
                "%zu-byte device scratch", R, vocab, need, size_t(DLLM_NOALLOC_SCRATCH_BYTES));
  hipStream_t s = static_cast<hipStream_t>(stream);
  int dev = -1;
  if (s) {
    TRY_HIP(hipStreamGetDevice(s, &dev), "hipStreamGetDevice");
  } else {
    TRY_HIP(hipGetDevice(&dev), "hipGetDevice");
  }
  void* ws = nullptr;
  dllm_status st = scratch_address(dev, &ws);
  if (st != DLLM_OK) return st;
  // every partial slot the merge reads is written by the partials kernel of
  // the same call: nothing in the scratch has to start at zero
  return vocab_entropy_topk(hidden, w_lm, R, d, vocab, dtype, row_scale, scale, mask_id, out, ws,
                            size_t(DLLM_NOALLOC_SCRATCH_BYTES), stream);
}

dllm_status rps_select_pivots(const dllm_stats* base, const int32_t* m_pos, int32_t n_m, const rps_params* prm,
                              rps_plan* plan, dllm_stream stream) {
  dllm_status st = check_stats(base, "base");
  if (st != DLLM_OK) return st;
  if (!m_pos || !prm || !plan) return fail(DLLM_EINVAL, "rps_select_pivots: NULL argument");
  if (n_m < 1 || n_m > RPS_MAX_MASKED) return fail(DLLM_ESHAPE, "n_m %d outside 1..%d", n_m, RPS_MAX_MASKED);
  if (prm->mode != RPS_PIVOT_PAPER && prm->mode != RPS_PIVOT_BAND) return fail(DLLM_EINVAL, "mode %d", prm->mode);
  if (prm->k_max < 1 || prm->k_max > base->k) return fail(DLLM_EINVAL, "k_max %d outside 1..k", prm->k_max);
  if (prm->n_cand < 1 || prm->n_cand > prm->k_max) return fail(DLLM_EINVAL, "n_cand %d outside 1..k_max", prm->n_cand);
  if (prm->n_pivots < 1 || prm->n_pivots > RPS_MAX_PIVOTS) return fail(DLLM_EINVAL, "n_pivots %d", prm->n_pivots);
  if (prm->max_branch < 1 || prm->max_branch > RPS_MAX_BRANCH) return fail(DLLM_EINVAL, "max_branch %d", prm->max_branch);
  if (!(prm->r >= 0.f) || !(prm->pct_lo >= 0.f) || !(prm->pct_hi <= 100.f) || !(prm->pct_lo <= prm->pct_hi) ||
      !std::isfinite(prm->tau_pivot))
    return fail(DLLM_EINVAL, "r / percentile / tau_pivot out of range");
  return hip_check(rps_select(to_out(*base), m_pos, n_m, *prm, plan, static_cast<hipStream_t>(stream)),
                   "rps_select_pivots");
}

dllm_status rps_build_branches(const int32_t* tokens, int32_t seq, const rps_plan* plan, int32_t anchor_first,
                               int32_t capacity, int32_t* out, dllm_stream stream) {
  if (!tokens || !plan || !out) return fail(DLLM_EINVAL, "rps_build_branches: NULL argument");
  if (seq < 1 || capacity < 1 || capacity > RPS_MAX_BRANCH + 1)
    return fail(DLLM_ESHAPE, "seq %d capacity %d", seq, capacity);
  return hip_check(rps_branches(tokens, seq, plan, anchor_first ? 1 : 0, capacity, out,
                                static_cast<hipStream_t>(stream)),
                   "rps_build_branches");
}

dllm_status rps_build_packed(const int32_t* tokens, int32_t seq, const rps_plan* plan, int32_t block_start,
                             int32_t block_len, int32_t capacity, int32_t* out, dllm_stream stream) {
  if (!tokens || !plan || !out) return fail(DLLM_EINVAL, "rps_build_packed: NULL argument");
  if (seq < 1 || capacity < 0 || capacity > RPS_MAX_BRANCH || block_len < 1 || block_start < 0 ||
      block_start + block_len > seq)
    return fail(DLLM_ESHAPE, "rps_build_packed: seq %d block %d..%d capacity %d", seq, block_start,
                block_start + block_len - 1, capacity);
  return hip_check(rps_branches_packed(tokens, seq, plan, block_start, block_len, capacity, out,
                                       static_cast<hipStream_t>(stream)),
                   "rps_build_packed");
}

dllm_status rps_lookahead_score(const dllm_stats* anchor, const dllm_stats* branches, int32_t branch_offset,
                                int32_t n_m, const rps_plan* plan, const float* anchor_logit, float lambda,
                                float* scores, float* deltas, rps_decision* dec, dllm_stream stream) {
  dllm_status st = check_stats(anchor, "anchor");
  if (st == DLLM_OK) st = check_stats(branches, "branches");
  if (st != DLLM_OK) return st;
  if (!plan || !dec) return fail(DLLM_EINVAL, "rps_lookahead_score: NULL plan or dec");
  if (n_m < 1 || n_m > RPS_MAX_MASKED) return fail(DLLM_ESHAPE, "n_m %d", n_m);
  if (branch_offset < 0 || branch_offset > 1) return fail(DLLM_EINVAL, "branch_offset %d", branch_offset);
  if (!(lambda >= 0.f) || !std::isfinite(lambda)) return fail(DLLM_EINVAL, "lambda must be finite and >= 0");
  return hip_check(rps_score(to_out(*anchor), to_out(*branches), branch_offset, n_m, plan, anchor_logit, lambda,
                             scores, deltas, dec, static_cast<hipStream_t>(stream)),
                   "rps_lookahead_score");
}

dllm_status rps_commit(int32_t* tokens, int32_t seq, int32_t* m_pos, int32_t n_m, const dllm_stats* base,
                       const rps_decision* dec,
                       const dllm_stats* branches, int32_t branch_offset, const dllm_stats* anchor, float tau,
                       int32_t* n_m_out, int32_t* committed, int32_t* n_committed, dllm_stream stream) {
  dllm_status st = check_stats(base, "base");
  if (st != DLLM_OK) return st;
  if (!tokens || !m_pos || !n_m_out || !committed || !n_committed)
    return fail(DLLM_EINVAL, "rps_commit: NULL argument");
  if (n_m < 1 || n_m > RPS_MAX_MASKED) return fail(DLLM_ESHAPE, "n_m %d", n_m);
  if (seq < 1) return fail(DLLM_ESHAPE, "seq %d", seq);
  if (dec) {
    st = check_stats(branches, "branches");
    if (st != DLLM_OK) return st;
    if (branches->k != base->k) return fail(DLLM_EINVAL, "branches.k != base.k");
    if (branch_offset < 0 || branch_offset > 1) return fail(DLLM_EINVAL, "branch_offset %d", branch_offset);
  }
  if (anchor) {
    st = check_stats(anchor, "anchor");
    if (st != DLLM_OK) return st;
    if (anchor->k != base->k) return fail(DLLM_EINVAL, "anchor.k != base.k");
  }
  if (std::isnan(tau)) return fail(DLLM_EINVAL, "tau is NaN");
  StatsOut bo = to_out(*base);
  StatsOut br = dec ? to_out(*branches) : StatsOut{};
  StatsOut an = anchor ? to_out(*anchor) : StatsOut{};
  return hip_check(rps_commit_step(tokens, seq, m_pos, n_m, bo, dec, dec ? &br : nullptr, branch_offset,
                                   anchor ? &an : nullptr, tau, n_m_out, committed, n_committed,
                                   static_cast<hipStream_t>(stream)),
                   "rps_commit");
}

dllm_status sched_commit(int32_t* tokens, int32_t seq, int32_t* m_pos, int32_t n_m, const dllm_stats* stats,
                         int32_t rule, int32_t k, int32_t* n_m_out, int32_t* committed, int32_t* n_committed,
                         dllm_stream stream) {
  dllm_status st = check_stats(stats, "stats");
  if (st != DLLM_OK) return st;
  if (!tokens || !m_pos || !n_m_out || !committed || !n_committed)
    return fail(DLLM_EINVAL, "sched_commit: NULL argument");
  if (rule != SCHED_TOP_CONFIDENCE && rule != SCHED_LOW_ENTROPY) return fail(DLLM_EINVAL, "rule %d", rule);
  if (k < 1) return fail(DLLM_EINVAL, "k %d", k);
  if (n_m < 1 || n_m > RPS_MAX_MASKED) return fail(DLLM_ESHAPE, "n_m %d", n_m);
  if (seq < 1) return fail(DLLM_ESHAPE, "seq %d", seq);
  return hip_check(sched_commit_step(tokens, seq, m_pos, n_m, to_out(*stats), rule, k, n_m_out, committed,
                                     n_committed, static_cast<hipStream_t>(stream)),
                   "sched_commit");
}

}  // extern "C"
