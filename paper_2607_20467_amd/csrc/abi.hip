// C-ABI entry points of libdcl: argument checks, packed-weight and workspace layouts, and the
// launch sequence of one denoising iteration (all asynchronous on the caller's stream).
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <new>
#include <vector>

#include "dcl_internal.h"

using namespace dcl;

namespace {

thread_local char g_err[512] = "";

dcl_status fail(dcl_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return s;
}

dcl_status hip_check(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(DCL_E_HIP, "%s: %s", what, hipGetErrorString(e));
  return DCL_OK;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

dcl_status check_config(const dcl_config* c) {
  if (!c) return fail(DCL_E_ARG, "config is NULL");
  if (c->n_layers < 1 || c->n_layers > 512) return fail(DCL_E_ARG, "n_layers %d outside [1, 512]", c->n_layers);
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(DCL_E_UNSUPPORTED, "head_dim %d: kernels exist for 64 and 128", c->head_dim);
  if (c->n_heads < 1 || c->n_kv_heads < 1 || c->n_heads % c->n_kv_heads != 0)
    return fail(DCL_E_UNSUPPORTED, "n_heads %d must be a positive multiple of n_kv_heads %d", c->n_heads,
                c->n_kv_heads);
  if (c->d_model < 16 || c->d_model % 16 != 0 || c->d_model > 8192)
    return fail(DCL_E_UNSUPPORTED, "d_model %d must be a multiple of 16, at most 8192", c->d_model);
  if (c->d_ffn < 16 || c->d_ffn % 16 != 0) return fail(DCL_E_UNSUPPORTED, "d_ffn %d must be a multiple of 16", c->d_ffn);
  if ((long)c->n_heads * c->head_dim > (1 << 20)) return fail(DCL_E_ARG, "n_heads * head_dim too large");
  if (c->vocab < 2) return fail(DCL_E_ARG, "vocab %d < 2", c->vocab);
  if (c->mask_id < 0 || c->mask_id >= c->vocab) return fail(DCL_E_ARG, "mask_id %d outside [0, vocab)", c->mask_id);
  if (!(c->rms_eps > 0.f) || !isfinite(c->rms_eps)) return fail(DCL_E_ARG, "rms_eps must be > 0");
  if (!(c->rope_base > 1.f) || !isfinite(c->rope_base)) return fail(DCL_E_ARG, "rope_base must be > 1");
  if (c->max_positions < 1 || c->max_positions > 65536)
    return fail(DCL_E_ARG, "max_positions %d outside [1, 65536]", c->max_positions);
  if (c->qkv_bias != 0 && c->qkv_bias != 1) return fail(DCL_E_ARG, "qkv_bias must be 0 or 1");
  if (c->rope_enabled != 0 && c->rope_enabled != 1) return fail(DCL_E_ARG, "rope_enabled must be 0 or 1");
  // the GEMM kernels form operand offsets (row * K) in 32 bits: every weight matrix stays below 2^31 elements
  const long d = c->d_model, hd = (long)c->n_heads * c->head_dim;
  const long qkv = (long)(c->n_heads + 2 * c->n_kv_heads) * c->head_dim;
  const long biggest = std::max({(long)c->vocab * d, qkv * d, hd * d, 2L * c->d_ffn * d});
  if (biggest >= (1L << 31))
    return fail(DCL_E_UNSUPPORTED, "a weight matrix of %ld elements: the kernels address at most 2^31", biggest);
  return DCL_OK;
}

WeightLayout make_layout(const dcl_config& c) {
  WeightLayout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align256(off + bytes);
    return o;
  };
  const size_t d = c.d_model, V = c.vocab, F = c.d_ffn, dh = c.head_dim;
  const size_t qkv = (size_t)(c.n_heads + 2 * c.n_kv_heads) * dh, hd = (size_t)c.n_heads * dh;
  L.embed = take(V * d * 2);
  for (int l = 0; l < c.n_layers; ++l) {
    LayerOffsets& o = L.layer[l];
    o.wqkv = take(qkv * d * 2);
    o.bqkv = take(qkv * 4);
    o.wo = take(d * hd * 2);
    o.wgu = take(2 * F * d * 2);
    o.wd = take(d * F * 2);
    o.g1 = take(d * 4);
    o.g2 = take(d * 4);
  }
  L.gf = take(d * 4);
  L.lm = take(V * d * 2);
  L.rope = take((size_t)c.max_positions * (dh / 2) * 8);
  L.total = off;
  return L;
}

StepLayout step_layout(const dcl_config& c, int B, int S, int P) {
  StepLayout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align256(off + bytes);
    return o;
  };
  const size_t T = (size_t)B * S, d = c.d_model, dh = c.head_dim;
  L.T = (int)T;
  L.S = S;
  L.koff = P > 0 ? P % 8 : 0;
  L.Sk = L.koff + S;
  L.Sp = (L.Sk + 7) / 8 * 8;
  L.n_vt = (c.vocab + kLmTile - 1) / kLmTile;
  L.r = take(T * d * 4);
  L.u = take(T * d * 2);
  L.q = take(T * c.n_heads * dh * 2);
  L.k = take((size_t)B * L.Sk * c.n_kv_heads * dh * 2);
  L.vt = take((size_t)B * c.n_kv_heads * dh * L.Sp * 2);
  L.o = take(T * c.n_heads * dh * 2);
  L.a = take(T * c.d_ffn * 2);
  L.rows = take(T * 4);
  L.count = take(4);
  L.hf = take(T * d * 2);
  const size_t np = T * L.n_vt * 4;
  L.pm1 = take(np);
  L.pi1 = take(np);
  L.pm2 = take(np);
  L.pi2 = take(np);
  L.ps = take(np);
  L.pt = take(np);
  // K-split slices of the residual GEMMs, folded into r by the next RMSNorm
  L.part = take((size_t)kMaxSplit * T * d * 4);
  L.total = off;
  return L;
}

template <class T>
T* at(void* base, size_t off) {
  return reinterpret_cast<T*>(reinterpret_cast<char*>(base) + off);
}

// ---------------------------------------------------------------- kernel-class timing
struct Profiler {
  bool on = false;
  struct Rec {
    int cls;
    hipEvent_t a, b;
  };
  std::vector<Rec> recs;
  std::vector<hipEvent_t> pool;
  int64_t launches[DCL_PROF_CLASSES] = {};
  double ms[DCL_PROF_CLASSES] = {};
  hipEvent_t get() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
  // fold completed records into the totals once many are pending (bounds the event count)
  void drain(bool wait) {
    for (Rec& r : recs) {
      if (wait) (void)hipEventSynchronize(r.b);
      float t = 0.f;
      if (hipEventElapsedTime(&t, r.a, r.b) == hipSuccess) {
        ms[r.cls] += t;
        launches[r.cls] += 1;
      }
      pool.push_back(r.a);
      pool.push_back(r.b);
    }
    recs.clear();
  }
};
Profiler g_prof;

struct ProfScope {
  hipStream_t s;
  int cls;
  hipEvent_t a = nullptr;
  ProfScope(int c, hipStream_t st) : s(st), cls(c) {
    if (!g_prof.on) return;
    if (g_prof.recs.size() > 8192) g_prof.drain(true);
    a = g_prof.get();
    if (a) (void)hipEventRecord(a, s);
  }
  ~ProfScope() {
    if (!a) return;
    hipEvent_t b = g_prof.get();
    if (!b) return;
    (void)hipEventRecord(b, s);
    g_prof.recs.push_back({cls, a, b});
  }
};
enum { P_EMBED, P_NORM, P_QKV, P_ATTN, P_O, P_GU, P_DOWN, P_COMPACT, P_LM, P_MERGE, P_SELECT };
#define PROF(cls) ProfScope prof_scope_##__LINE__(cls, s)

// Sizes, ranges and the cache description (host-only, no device access). Every check that depends
// only on the arguments comes before the state check, so a call with bad sizes is reported as such
// whether or not weights were loaded.
dcl_status check_shape_args(const Model* m, int32_t B, int32_t S, const dcl_kv* kv) {
  if (!m) return fail(DCL_E_ARG, "model is NULL");
  if (B < 1 || S < 1) return fail(DCL_E_ARG, "B=%d, S=%d must be >= 1", B, S);
  if ((long)B * S > (1 << 22)) return fail(DCL_E_ARG, "B*S = %ld too large", (long)B * S);
  // the QKV epilogue addresses q/k/v^T with 32 bits; a ragged cached prefix adds up to 7 carried keys (and
  // their padding) per sequence
  const int pad = (kv && kv->prefix_len % 8 != 0) ? 16 : 8;
  if ((long)B * (S + pad) * m->qkv_rows() >= (1L << 31))
    return fail(DCL_E_UNSUPPORTED, "B*S = %ld tokens: q/k/v would reach 2^31 elements", (long)B * S);
  // the GEMMs address their activation operand ([tokens, K], K up to max(d_model, H*dh, d_ffn)) with 32 bits
  const long kmax = std::max({(long)m->cfg.d_model, (long)m->cfg.n_heads * m->cfg.head_dim, (long)m->cfg.d_ffn});
  if ((long)B * S * kmax >= (1L << 31))
    return fail(DCL_E_UNSUPPORTED, "B*S = %ld tokens: a GEMM activation operand would reach 2^31 elements",
                (long)B * S);
  const int P = kv ? kv->prefix_len : 0;
  if (kv) {
    if (!kv->k || !kv->v) return fail(DCL_E_ARG, "kv->k / kv->v is NULL");
    if (P < 0) return fail(DCL_E_ARG, "kv prefix_len %d must be >= 0", P);
    const int cap = kv->capacity ? kv->capacity : P;
    if (cap < P || cap % 8 != 0)
      return fail(DCL_E_ARG, "kv capacity %d must be a multiple of 8 and >= prefix_len %d", kv->capacity, P);
    for (int l = 0; l < m->cfg.n_layers; ++l)
      if (P > 0 && (!kv->k[l] || !kv->v[l])) return fail(DCL_E_ARG, "kv cache pointer of layer %d is NULL", l);
  }
  if ((long)P + S > m->cfg.max_positions)
    return fail(DCL_E_ARG, "positions up to %ld exceed max_positions %d", (long)P + S, m->cfg.max_positions);
  return DCL_OK;
}

dcl_status check_workspace(const Model* m, int32_t B, int32_t S, int32_t P, void* ws, size_t ws_bytes) {
  if (!ws) return fail(DCL_E_ARG, "workspace is NULL");
  if ((reinterpret_cast<uintptr_t>(ws) & 255) != 0) return fail(DCL_E_ARG, "workspace must be 256-byte aligned");
  const size_t need = step_layout(m->cfg, B, S, P).total;
  if (ws_bytes < need) return fail(DCL_E_WORKSPACE, "workspace %zu bytes < required %zu", ws_bytes, need);
  return DCL_OK;
}

dcl_status check_step_args(const Model* m, const int32_t* tokens, int32_t B, int32_t S, const dcl_kv* kv, void* ws,
                           size_t ws_bytes) {
  dcl_status st = check_shape_args(m, B, S, kv);
  if (st != DCL_OK) return st;
  if (!tokens) return fail(DCL_E_ARG, "tokens is NULL");
  if (!m->loaded) return fail(DCL_E_STATE, "weights not loaded");
  return check_workspace(m, B, S, kv ? kv->prefix_len : 0, ws, ws_bytes);
}

// Device-to-device copy of a stage's result into a caller buffer (test support; null = not wanted).
void tap(void* dst, const void* src, size_t bytes, hipStream_t s) {
  if (dst) (void)hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, s);
}

// a3-a7 for layer l on the residual stream in ws.r. `pending` is the number of K-split slices of the
// previous residual GEMM still to be added to ws.r (the first RMSNorm folds them in); the return value
// is that number for this layer's down projection. With `writeback` the layer's fresh keys/values go
// into the cache and the layer stops after them (returns -1). With `taps` every intermediate is also
// copied out, and the down projection's slices are folded into ws.r before r_out is copied.
int run_layer(const Model* m, int l, int B, int S, const dcl_kv* kv, void* ws, const StepLayout& L, hipStream_t s,
              int pending, bool writeback = false, const dcl_layer_taps* taps = nullptr) {
  const dcl_config& c = m->cfg;
  const int T = B * S, d = c.d_model, dh = c.head_dim;
  const int P = kv ? kv->prefix_len : 0;
  void* wb = m->wbuf;
  float* r = at<float>(ws, L.r);
  bf16_t* u = at<bf16_t>(ws, L.u);
  bf16_t* a = at<bf16_t>(ws, L.a);
  bf16_t* o = at<bf16_t>(ws, L.o);
  float* part = at<float>(ws, L.part);
  const LayerOffsets& lo = m->lay.layer[l];
  {
    PROF(P_NORM);
    launch_rmsnorm(r, at<float>(wb, lo.g1), u, T, d, c.rms_eps, nullptr, nullptr, part, pending, s);
  }
  if (taps) tap(taps->u, u, (size_t)T * d * 2, s);
  QkvOut qo;
  qo.q = at<bf16_t>(ws, L.q);
  qo.k = at<bf16_t>(ws, L.k);
  qo.vt = at<bf16_t>(ws, L.vt);
  qo.bias = c.qkv_bias ? at<float>(wb, lo.bqkv) : nullptr;
  qo.rope = c.rope_enabled ? at<float2>(wb, m->lay.rope) : nullptr;
  qo.H = c.n_heads;
  qo.Hkv = c.n_kv_heads;
  qo.dh = dh;
  qo.S = S;
  qo.Sp = L.Sp;
  qo.Sk = L.Sk;
  qo.koff = L.koff;
  qo.pos0 = P;
  {
    PROF(P_QKV);
    gemm_qkv(at<bf16_t>(wb, lo.wqkv), u, m->qkv_rows(), T, d, qo, s);
  }
  const int Pc = kv ? (kv->capacity ? kv->capacity : P) : 0;
  if (kv && L.koff > 0)  // the newest P mod 8 cached keys/values in front of the fresh ones
    launch_kv_carry(static_cast<const bf16_t*>(kv->k[l]), static_cast<const bf16_t*>(kv->v[l]), qo.k, qo.vt, B,
                    c.n_kv_heads, L.Sk, L.Sp, dh, P, Pc, s);
  if (taps) {
    tap(taps->q, qo.q, (size_t)T * c.n_heads * dh * 2, s);
    tap(taps->k, qo.k, (size_t)B * L.Sk * c.n_kv_heads * dh * 2, s);
    tap(taps->v, qo.vt, (size_t)B * c.n_kv_heads * dh * L.Sp * 2, s);
  }
  if (writeback) {  // this layer's fresh keys and values into the cache at [P, P + S)
    launch_kv_writeback(qo.k, qo.vt, static_cast<bf16_t*>(const_cast<void*>(kv->k[l])),
                        static_cast<bf16_t*>(const_cast<void*>(kv->v[l])), B, c.n_kv_heads, S, L.Sk, L.Sp, L.koff,
                        dh, P, Pc, s);
    if (l == c.n_layers - 1) return -1;  // nothing after the last layer's keys and values is needed
  }
  AttnArgs aa;
  aa.q = qo.q;
  aa.k = qo.k;
  aa.vt = qo.vt;
  aa.kc = (kv && P - L.koff > 0) ? static_cast<const bf16_t*>(kv->k[l]) : nullptr;
  aa.vc = (kv && P - L.koff > 0) ? static_cast<const bf16_t*>(kv->v[l]) : nullptr;
  aa.o = o;
  aa.B = B;
  aa.H = c.n_heads;
  aa.Hkv = c.n_kv_heads;
  aa.dh = dh;
  aa.S = S;
  aa.Sp = L.Sp;
  aa.Sk = L.Sk;
  aa.P = P - L.koff;  // whole 8-key chunks of the cache; the rest was carried into the fresh buffers
  aa.Pc = Pc;
  aa.scale_log2 = (float)(1.4426950408889634 / sqrt((double)dh));
  {
    PROF(P_ATTN);
    launch_attention(aa, s);
  }
  if (taps) tap(taps->o, o, (size_t)T * c.n_heads * dh * 2, s);
  {
    PROF(P_O);
    pending = gemm_resid(at<bf16_t>(wb, lo.wo), o, d, T, c.n_heads * dh, r, part, s);
  }
  {
    PROF(P_NORM);
    launch_rmsnorm(r, at<float>(wb, lo.g2), u, T, d, c.rms_eps, nullptr, nullptr, part, pending, s);
  }
  if (taps) {
    tap(taps->r_mid, r, (size_t)T * d * 4, s);
    tap(taps->u2, u, (size_t)T * d * 2, s);
  }
  {
    PROF(P_GU);
    gemm_swiglu(at<bf16_t>(wb, lo.wgu), u, 2 * c.d_ffn, T, d, a, s);
  }
  if (taps) tap(taps->a, a, (size_t)T * c.d_ffn * 2, s);
  {
    PROF(P_DOWN);
    pending = gemm_resid(at<bf16_t>(wb, lo.wd), a, d, T, c.d_ffn, r, part, s);
  }
  if (taps) {
    // fold the down projection's slices into r exactly as the next RMSNorm would (same kernel, same
    // split order); its normalised output goes to the h_f scratch and is not used
    if (pending > 0)
      launch_rmsnorm(r, at<float>(wb, m->lay.gf), at<bf16_t>(ws, L.hf), T, d, c.rms_eps, nullptr, nullptr, part,
                     pending, s);
    pending = 0;
    tap(taps->r_out, r, (size_t)T * d * 4, s);
  }
  return pending;
}

// a2-a7: embedding and every transformer layer. Returns the number of K-split slices of the last
// residual GEMM still to be added to ws.r (the final RMSNorm folds them in).
int run_forward(const Model* m, const int32_t* tokens, int B, int S, const dcl_kv* kv, void* ws,
                const StepLayout& L, hipStream_t s, bool writeback = false) {
  const dcl_config& c = m->cfg;
  int pending = 0;  // K-split slices of the last residual GEMM not yet added to r
  {
    PROF(P_EMBED);
    launch_embed(tokens, at<bf16_t>(m->wbuf, m->lay.embed), at<float>(ws, L.r), B * S, c.d_model, c.vocab, s);
  }
  for (int l = 0; l < c.n_layers; ++l) {
    pending = run_layer(m, l, B, S, kv, ws, L, s, pending, writeback);
    if (pending < 0) return 0;
  }
  return pending;
}

dcl_status check_denoise_args(const Model* m, const int32_t* tokens, int32_t B, int32_t S, const int32_t* p,
                              int32_t gen_end, const dcl_kv* kv, uint32_t flags, const dcl_row_stats& out, void* ws,
                              size_t ws_bytes) {
  dcl_status st = check_step_args(m, tokens, B, S, kv, ws, ws_bytes);
  if (st != DCL_OK) return st;
  if (!p) return fail(DCL_E_ARG, "p is NULL");
  if (gen_end < 0 || gen_end > S) return fail(DCL_E_ARG, "gen_end %d outside [0, S=%d]", gen_end, S);
  if (flags & ~(uint32_t)(DCL_SCORE_ALL_UNCOMMITTED | DCL_SCORE_SUPPRESS_MASK))
    return fail(DCL_E_ARG, "unknown flags 0x%x", flags);
  if (!out.top1 || !out.top2 || !out.conf || !out.p2 || !out.lse) return fail(DCL_E_ARG, "an output array is NULL");
  return DCL_OK;
}

// a2-a10 on `stream` (arguments already checked).
void enqueue_denoise(const Model* m, const int32_t* tokens, int32_t B, int32_t S, const int32_t* p, int32_t gen_end,
                     const dcl_kv* kv, uint32_t flags, const dcl_row_stats& out, void* ws, hipStream_t stream) {
  const dcl_config& c = m->cfg;
  const StepLayout L = step_layout(c, B, S, kv ? kv->prefix_len : 0);
  const int pending = run_forward(m, tokens, B, S, kv, ws, L, stream);
  int32_t* rows = at<int32_t>(ws, L.rows);
  int32_t* count = at<int32_t>(ws, L.count);
  hipStream_t s = stream;
  {
    PROF(P_COMPACT);
    launch_compact(tokens, p, B, S, gen_end, c.mask_id, (flags & DCL_SCORE_ALL_UNCOMMITTED) ? 1 : 0, rows, count, out,
                   stream);
  }
  bf16_t* hf = at<bf16_t>(ws, L.hf);
  {
    PROF(P_NORM);
    launch_rmsnorm(at<float>(ws, L.r), at<float>(m->wbuf, m->lay.gf), hf, L.T, c.d_model, c.rms_eps, rows, count,
                   at<float>(ws, L.part), pending, stream);
  }
  LmOut lo;
  lo.pm1 = at<float>(ws, L.pm1);
  lo.pi1 = at<int32_t>(ws, L.pi1);
  lo.pm2 = at<float>(ws, L.pm2);
  lo.pi2 = at<int32_t>(ws, L.pi2);
  lo.ps = at<float>(ws, L.ps);
  lo.pt = at<float>(ws, L.pt);
  lo.n_vt = L.n_vt;
  lo.count = count;
  lo.exclude = (flags & DCL_SCORE_SUPPRESS_MASK) ? c.mask_id : -1;
  {
    PROF(P_LM);
    gemm_lmhead(at<bf16_t>(m->wbuf, m->lay.lm), hf, c.vocab, L.T, c.d_model, lo, stream);
  }
  {
    PROF(P_MERGE);
    launch_merge(lo.pm1, lo.pi1, lo.pm2, lo.pi2, lo.ps, lo.pt, L.n_vt, rows, count, L.T, out, stream);
  }
}

dcl_status check_select_args(const int32_t* tokens, int32_t B, int32_t S, const int32_t* p, int32_t gen_end,
                             int32_t L, int32_t block_origin, int32_t block_len, float tau_commit, float tau_draft,
                             const dcl_row_stats& in, uint32_t flags) {
  if (!tokens || !p) return fail(DCL_E_ARG, "tokens / p is NULL");
  if (!in.top1 || !in.conf) return fail(DCL_E_ARG, "in.top1 / in.conf is NULL");
  if ((flags & DCL_SEL_MARGIN) && !in.p2) return fail(DCL_E_ARG, "DCL_SEL_MARGIN needs in.p2");
  if (B < 1 || S < 1) return fail(DCL_E_ARG, "B=%d, S=%d must be >= 1", B, S);
  if (gen_end < 0 || gen_end > S) return fail(DCL_E_ARG, "gen_end %d outside [0, S=%d]", gen_end, S);
  if (L < 1) return fail(DCL_E_ARG, "window L=%d must be >= 1", L);
  if (block_len < 0) return fail(DCL_E_ARG, "block_len %d must be >= 0", block_len);
  if (block_len > 0 && (block_origin < 0 || block_origin > S))
    return fail(DCL_E_ARG, "block_origin %d outside [0, S=%d]", block_origin, S);
  if (!(tau_commit >= 0.f && tau_commit <= 1.f)) return fail(DCL_E_ARG, "tau_commit %g outside [0, 1]", tau_commit);
  if (!(tau_draft >= 0.f) || isnan(tau_draft)) return fail(DCL_E_ARG, "tau_draft %g must be >= 0", tau_draft);
  if (flags & ~(uint32_t)(DCL_SEL_NO_PROGRESS_GUARD | DCL_SEL_SCORE_ALL | DCL_SEL_NONCONTIGUOUS |
                          DCL_SEL_CONTIGUOUS_DRAFTS | DCL_SEL_MARGIN))
    return fail(DCL_E_ARG, "unknown flags 0x%x", flags);
  if ((flags & DCL_SEL_NONCONTIGUOUS) && (flags & (DCL_SEL_SCORE_ALL | DCL_SEL_CONTIGUOUS_DRAFTS)))
    return fail(DCL_E_ARG, "DCL_SEL_NONCONTIGUOUS takes no draft or score-all flag (flags 0x%x)", flags);
  return DCL_OK;
}

// Scratch of dcl_denoise_step_noalloc: a fixed device array in the library's code object, one copy per
// device (each device that runs the call holds it until the process ends). Host code never uses the
// array's name as an address: the device address comes from hipGetSymbolAddress, taken once per device
// with that device current, and kernels receive that address as their workspace pointer.
static __device__ __align__(256) unsigned char scratch[DCL_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

// Device address of the current device's scratch (looked up on the first call per device).
dcl_status scratch_address(void** out) {
  int dev = -1;
  dcl_status st = hip_check(hipGetDevice(&dev), "hipGetDevice");
  if (st != DCL_OK) return st;
  if (dev < 0 || dev >= kMaxDevices) return fail(DCL_E_UNSUPPORTED, "device %d: at most %d devices", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    st = hip_check(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
    if (st != DCL_OK) return st;
    if (!p || (reinterpret_cast<uintptr_t>(p) & 255) != 0) return fail(DCL_E_HIP, "scratch address %p not 256-byte aligned", p);
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return DCL_OK;
}

}  // namespace

extern "C" {

const char* dcl_status_string(dcl_status s) {
  switch (s) {
    case DCL_OK: return "ok";
    case DCL_E_ARG: return "invalid argument";
    case DCL_E_UNSUPPORTED: return "unsupported geometry";
    case DCL_E_WORKSPACE: return "buffer too small";
    case DCL_E_HIP: return "HIP error";
    case DCL_E_STATE: return "invalid state";
  }
  return "unknown status";
}

const char* dcl_last_error(void) { return g_err; }

dcl_status dcl_model_create(const dcl_config* cfg, dcl_model_t* out) {
  if (!out) return fail(DCL_E_ARG, "out is NULL");
  *out = nullptr;
  dcl_status st = check_config(cfg);
  if (st != DCL_OK) return st;
  Model* m = new (std::nothrow) Model();
  if (!m) return fail(DCL_E_ARG, "out of host memory");
  m->cfg = *cfg;
  m->lay = make_layout(*cfg);
  *out = reinterpret_cast<dcl_model_t>(m);
  return DCL_OK;
}

void dcl_model_destroy(dcl_model_t model) { delete reinterpret_cast<Model*>(model); }

size_t dcl_weights_bytes(const dcl_config* cfg) {
  if (check_config(cfg) != DCL_OK) return 0;
  return make_layout(*cfg).total;
}

dcl_status dcl_load_weights(dcl_model_t model, void* dev_buf, size_t bytes, const void* const* src, int32_t n_src,
                            int32_t src_dtype, hipStream_t stream) {
  Model* m = reinterpret_cast<Model*>(model);
  if (!m) return fail(DCL_E_ARG, "model is NULL");
  if (!dev_buf || !src) return fail(DCL_E_ARG, "dev_buf / src is NULL");
  if ((reinterpret_cast<uintptr_t>(dev_buf) & 255) != 0) return fail(DCL_E_ARG, "dev_buf must be 256-byte aligned");
  if (bytes < m->lay.total) return fail(DCL_E_WORKSPACE, "weight buffer %zu bytes < required %zu", bytes, m->lay.total);
  if (src_dtype != DCL_DTYPE_F32 && src_dtype != DCL_DTYPE_BF16) return fail(DCL_E_ARG, "src_dtype %d", src_dtype);
  const dcl_config& c = m->cfg;
  const int expect = 1 + 12 * c.n_layers + 2;
  if (n_src != expect) return fail(DCL_E_ARG, "n_src %d, expected %d", n_src, expect);
  for (int i = 0; i < n_src; ++i) {
    const int li = (i - 1) % 12;
    const bool is_bias = i >= 1 && i < 1 + 12 * c.n_layers && li >= 3 && li <= 5;
    if (!src[i] && !(is_bias && !c.qkv_bias)) return fail(DCL_E_ARG, "src[%d] is NULL", i);
  }
  const size_t es = src_dtype == DCL_DTYPE_F32 ? 4 : 2;
  const size_t d = c.d_model, V = c.vocab, F = c.d_ffn, dh = c.head_dim, H = c.n_heads, Hkv = c.n_kv_heads;
  size_t biggest = V * d;
  if (F * d > biggest) biggest = F * d;
  if (H * dh * d > biggest) biggest = H * dh * d;
  void* stage = nullptr;
  dcl_status st = hip_check(hipMalloc(&stage, biggest * es), "hipMalloc(staging)");
  if (st != DCL_OK) return st;
  void* wb = dev_buf;
  auto put_mat = [&](const void* p, size_t rows, size_t cols, size_t dst_off, int mode, int dst_row0) -> dcl_status {
    dcl_status e = hip_check(hipMemcpyAsync(stage, p, rows * cols * es, hipMemcpyDefault, stream), "hipMemcpyAsync");
    if (e != DCL_OK) return e;
    launch_pack_rows(stage, src_dtype, at<bf16_t>(wb, dst_off), (int)rows, (int)cols, mode, (int)dh, dst_row0, stream);
    return hip_check(hipGetLastError(), "pack_rows launch");
  };
  auto put_vec = [&](const void* p, size_t n, size_t dst_off, int mode, int dst0) -> dcl_status {
    if (p) {
      dcl_status e = hip_check(hipMemcpyAsync(stage, p, n * es, hipMemcpyDefault, stream), "hipMemcpyAsync");
      if (e != DCL_OK) return e;
    }
    launch_pack_vec(p ? stage : nullptr, src_dtype, at<float>(wb, dst_off), (int)n, mode, (int)dh, dst0, stream);
    return hip_check(hipGetLastError(), "pack_vec launch");
  };
#define TRY(x)            \
  do {                    \
    st = (x);             \
    if (st != DCL_OK) {   \
      (void)hipFree(stage); \
      return st;          \
    }                     \
  } while (0)
  TRY(put_mat(src[0], V, d, m->lay.embed, 0, 0));
  for (int l = 0; l < c.n_layers; ++l) {
    const void* const* s = src + 1 + 12 * l;
    const LayerOffsets& lo = m->lay.layer[l];
    TRY(put_mat(s[0], H * dh, d, lo.wqkv, 1, 0));
    TRY(put_mat(s[1], Hkv * dh, d, lo.wqkv, 1, (int)(H * dh)));
    TRY(put_mat(s[2], Hkv * dh, d, lo.wqkv, 0, (int)((H + Hkv) * dh)));
    TRY(put_vec(c.qkv_bias ? s[3] : nullptr, H * dh, lo.bqkv, 1, 0));
    TRY(put_vec(c.qkv_bias ? s[4] : nullptr, Hkv * dh, lo.bqkv, 1, (int)(H * dh)));
    TRY(put_vec(c.qkv_bias ? s[5] : nullptr, Hkv * dh, lo.bqkv, 0, (int)((H + Hkv) * dh)));
    TRY(put_mat(s[6], d, H * dh, lo.wo, 0, 0));
    TRY(put_mat(s[7], F, d, lo.wgu, 2, 0));
    TRY(put_mat(s[8], F, d, lo.wgu, 3, 0));
    TRY(put_mat(s[9], d, F, lo.wd, 0, 0));
    TRY(put_vec(s[10], d, lo.g1, 0, 0));
    TRY(put_vec(s[11], d, lo.g2, 0, 0));
  }
  TRY(put_vec(src[1 + 12 * c.n_layers], d, m->lay.gf, 0, 0));
  TRY(put_mat(src[2 + 12 * c.n_layers], V, d, m->lay.lm, 0, 0));
#undef TRY
  // RoPE table: theta = pos * base^(-2i/dh), built in float64 on the host, stored as float32 (cos, sin).
  const size_t half = dh / 2, npos = (size_t)c.max_positions;
  std::vector<float> tab(npos * half * 2);
  for (size_t pos = 0; pos < npos; ++pos)
    for (size_t i = 0; i < half; ++i) {
      const double inv_freq = pow((double)c.rope_base, -(2.0 * (double)i) / (double)dh);
      const double ang = (double)pos * inv_freq;
      tab[(pos * half + i) * 2] = (float)cos(ang);
      tab[(pos * half + i) * 2 + 1] = (float)sin(ang);
    }
  st = hip_check(hipMemcpyAsync(at<char>(wb, m->lay.rope), tab.data(), tab.size() * 4, hipMemcpyHostToDevice, stream),
                 "hipMemcpyAsync(rope)");
  dcl_status st2 = hip_check(hipStreamSynchronize(stream), "hipStreamSynchronize(load)");
  (void)hipFree(stage);
  if (st != DCL_OK) return st;
  if (st2 != DCL_OK) return st2;
  m->wbuf = dev_buf;
  m->loaded = true;
  return DCL_OK;
}

size_t dcl_workspace_bytes(dcl_model_t model, int32_t B, int32_t S, int32_t kv_prefix) {
  Model* m = reinterpret_cast<Model*>(model);
  if (!m || B < 1 || S < 1 || kv_prefix < 0 || (long)B * S > (1 << 22)) return 0;
  return step_layout(m->cfg, B, S, kv_prefix).total;
}


dcl_status dcl_denoise_step(dcl_model_t model, const int32_t* tokens, int32_t B, int32_t S, const int32_t* p,
                            int32_t gen_end, const dcl_kv* kv, uint32_t flags, dcl_row_stats out, void* ws,
                            size_t ws_bytes, hipStream_t stream) {
  Model* m = reinterpret_cast<Model*>(model);
  dcl_status st = check_denoise_args(m, tokens, B, S, p, gen_end, kv, flags, out, ws, ws_bytes);
  if (st != DCL_OK) return st;
  (void)hipGetLastError();  // clear a stale error so the check below reports this call's launches
  enqueue_denoise(m, tokens, B, S, p, gen_end, kv, flags, out, ws, stream);
  return hip_check(hipGetLastError(), "denoise_step launch");
}
dcl_status dcl_denoise_step_noalloc(dcl_model_t model, const int32_t* tokens, int32_t B, int32_t S, const int32_t* p,
                                    int32_t gen_end, const dcl_kv* kv, uint32_t flags, dcl_row_stats out,
                                    hipStream_t stream) {
  Model* m = reinterpret_cast<Model*>(model);
  dcl_status st = check_shape_args(m, B, S, kv);
  if (st != DCL_OK) return st;
  const size_t need = step_layout(m->cfg, B, S, kv ? kv->prefix_len : 0).total;
  if (need > (size_t)DCL_NOALLOC_SCRATCH_BYTES)
    return fail(DCL_E_WORKSPACE, "B=%d, S=%d needs %zu bytes of scratch; the static scratch holds %zu (use "
                "dcl_denoise_step with a workspace)", B, S, need, (size_t)DCL_NOALLOC_SCRATCH_BYTES);
  if (!m->loaded) return fail(DCL_E_STATE, "weights not loaded");
  void* ws = nullptr;
  st = scratch_address(&ws);
  if (st != DCL_OK) return st;
  st = check_denoise_args(m, tokens, B, S, p, gen_end, kv, flags, out, ws, (size_t)DCL_NOALLOC_SCRATCH_BYTES);
  if (st != DCL_OK) return st;
  (void)hipGetLastError();
  enqueue_denoise(m, tokens, B, S, p, gen_end, kv, flags, out, ws, stream);
  return hip_check(hipGetLastError(), "denoise_step_noalloc launch");
}

dcl_status dcl_select_contiguous(int32_t* tokens, int32_t B, int32_t S, int32_t* p, int32_t gen_end, int32_t L,
                                 int32_t block_origin, int32_t block_len, float tau_commit, float tau_draft,
                                 int32_t mask_id, dcl_row_stats in, int32_t* K_raw, int32_t* K_eff, uint32_t flags,
                                 hipStream_t stream) {
  dcl_status st = check_select_args(tokens, B, S, p, gen_end, L, block_origin, block_len, tau_commit, tau_draft, in,
                                    flags);
  if (st != DCL_OK) return st;
  (void)hipGetLastError();
  {
    hipStream_t s = stream;
    PROF(P_SELECT);
    launch_select(tokens, B, S, p, gen_end, L, block_origin, block_len, tau_commit, tau_draft, mask_id, in, K_raw,
                  K_eff, flags, stream);
  }
  return hip_check(hipGetLastError(), "select launch");
}

dcl_status dcl_generate(dcl_model_t model, int32_t* tokens, int32_t B, int32_t S, int32_t* p, int32_t gen_end,
                        const dcl_kv* kv, uint32_t score_flags, int32_t L, int32_t block_origin,
                        int32_t block_len, float tau_commit, float tau_draft, uint32_t select_flags, int32_t max_steps,
                        int32_t check_every, dcl_row_stats stats, int32_t* K_raw, int32_t* K_eff, int32_t* k_hist,
                        void* ws, size_t ws_bytes, int32_t* steps_out, hipStream_t stream) {
  Model* m = reinterpret_cast<Model*>(model);
  dcl_status st = check_denoise_args(m, tokens, B, S, p, gen_end, kv, score_flags, stats, ws, ws_bytes);
  if (st != DCL_OK) return st;
  st = check_select_args(tokens, B, S, p, gen_end, L, block_origin, block_len, tau_commit, tau_draft, stats,
                         select_flags);
  if (st != DCL_OK) return st;
  if (max_steps < 1 || check_every < 1) return fail(DCL_E_ARG, "max_steps %d and check_every %d must be >= 1",
                                                    max_steps, check_every);
  if (!steps_out) return fail(DCL_E_ARG, "steps_out is NULL");
  *steps_out = 0;
  const int mask_id = m->cfg.mask_id;
  (void)hipGetLastError();

  // A private stream (the caller's may be the legacy null stream, which cannot be captured),
  // ordered after the caller's stream on entry and before it on return.
  hipStream_t gs = nullptr;
  hipEvent_t ev = nullptr;
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
  std::vector<int32_t> ph(B);
  int n = 0;
  bool done = false;
  auto iteration = [&](hipStream_t q) {
    enqueue_denoise(m, tokens, B, S, p, gen_end, kv, score_flags, stats, ws, q);
    hipStream_t s = q;
    PROF(P_SELECT);
    launch_select(tokens, B, S, p, gen_end, L, block_origin, block_len, tau_commit, tau_draft, mask_id, stats, K_raw,
                  K_eff, select_flags, q, k_hist);
  };
  auto check = [&]() -> dcl_status {  // host copy of p: done when every sequence reached gen_end
    dcl_status e = hip_check(hipMemcpyAsync(ph.data(), p, (size_t)B * sizeof(int32_t), hipMemcpyDeviceToHost, gs),
                             "hipMemcpyAsync(p)");
    if (e == DCL_OK) e = hip_check(hipStreamSynchronize(gs), "hipStreamSynchronize");
    if (e != DCL_OK) return e;
    done = true;
    for (int b = 0; b < B; ++b) done = done && (ph[b] < 0 || ph[b] >= gen_end);
    return DCL_OK;
  };
  st = hip_check(hipStreamCreateWithFlags(&gs, hipStreamNonBlocking), "hipStreamCreateWithFlags");
  if (st == DCL_OK) st = hip_check(hipEventCreateWithFlags(&ev, hipEventDisableTiming), "hipEventCreate");
  if (st == DCL_OK) st = hip_check(hipEventRecord(ev, stream), "hipEventRecord");
  if (st == DCL_OK) st = hip_check(hipStreamWaitEvent(gs, ev, 0), "hipStreamWaitEvent");
  if (st == DCL_OK) {
    // Algorithm 1's loop-top draft invalidation for the first iteration; later ones end with it
    launch_remask(tokens, B, S, p, gen_end, L, block_origin, block_len, mask_id, gs);
    st = check();
  }
  // The first iteration runs eagerly (it also performs every one-time kernel set-up, which must not
  // happen under capture); later ones replay one captured iteration. With kernel-class profiling on,
  // every iteration runs eagerly so each launch keeps its event pair.
  while (st == DCL_OK && !done && n < max_steps) {
    if (n > 0 && !exec && !g_prof.on) {
      st = hip_check(hipStreamBeginCapture(gs, hipStreamCaptureModeThreadLocal), "hipStreamBeginCapture");
      if (st != DCL_OK) break;
      iteration(gs);
      const hipError_t launch_err = hipGetLastError();
      st = hip_check(hipStreamEndCapture(gs, &graph), "hipStreamEndCapture");
      if (st == DCL_OK) st = hip_check(launch_err, "captured iteration launch");
      if (st == DCL_OK) st = hip_check(hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0), "hipGraphInstantiate");
      if (st != DCL_OK) break;
    }
    if (exec) st = hip_check(hipGraphLaunch(exec, gs), "hipGraphLaunch");
    else {
      iteration(gs);
      st = hip_check(hipGetLastError(), "iteration launch");
    }
    if (st != DCL_OK) break;
    ++n;
    if (n % check_every == 0 || n == max_steps) st = check();
  }
  *steps_out = n;
  if (gs) {
    if (st == DCL_OK) st = hip_check(hipEventRecord(ev, gs), "hipEventRecord");
    if (st == DCL_OK) st = hip_check(hipStreamWaitEvent(stream, ev, 0), "hipStreamWaitEvent");
    (void)hipStreamSynchronize(gs);
  }
  if (exec) (void)hipGraphExecDestroy(exec);
  if (graph) (void)hipGraphDestroy(graph);
  if (ev) (void)hipEventDestroy(ev);
  if (gs) (void)hipStreamDestroy(gs);
  return st;
}

dcl_status dcl_kv_append(dcl_model_t model, const int32_t* tokens, int32_t B, int32_t S, const dcl_kv* kv, void* ws,
                         size_t ws_bytes, hipStream_t stream) {
  Model* m = reinterpret_cast<Model*>(model);
  if (!kv) return fail(DCL_E_ARG, "kv is NULL");
  dcl_status st = check_step_args(m, tokens, B, S, kv, ws, ws_bytes);
  if (st != DCL_OK) return st;
  for (int l = 0; l < m->cfg.n_layers; ++l)
    if (!kv->k[l] || !kv->v[l]) return fail(DCL_E_ARG, "kv cache pointer of layer %d is NULL", l);
  const int cap = kv->capacity ? kv->capacity : kv->prefix_len;
  if ((long)kv->prefix_len + S > cap)
    return fail(DCL_E_ARG, "prefix_len %d + S %d exceeds the cache capacity %d", kv->prefix_len, S, cap);
  (void)hipGetLastError();
  run_forward(m, tokens, B, S, kv, ws, step_layout(m->cfg, B, S, kv->prefix_len), stream, true);
  return hip_check(hipGetLastError(), "kv_append launch");
}

struct ScoreLayout {
  size_t rows, count, pm1, pi1, pm2, pi2, ps, pt, total;
  int n_vt;
};

static ScoreLayout score_layout(const dcl_config& c, int n) {
  ScoreLayout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align256(off + bytes);
    return o;
  };
  L.n_vt = (c.vocab + kLmTile - 1) / kLmTile;
  L.rows = take((size_t)n * 4);
  L.count = take(4);
  const size_t np = (size_t)n * L.n_vt * 4;
  L.pm1 = take(np);
  L.pi1 = take(np);
  L.pm2 = take(np);
  L.pi2 = take(np);
  L.ps = take(np);
  L.pt = take(np);
  L.total = off;
  return L;
}

size_t dcl_score_workspace_bytes(dcl_model_t model, int32_t n) {
  Model* m = reinterpret_cast<Model*>(model);
  if (!m || n < 1 || n > (1 << 22)) return 0;
  return score_layout(m->cfg, n).total;
}

dcl_status dcl_score_hidden(dcl_model_t model, const void* hidden, int32_t n, dcl_row_stats out, void* ws,
                            size_t ws_bytes, hipStream_t stream) {
  Model* m = reinterpret_cast<Model*>(model);
  if (!m) return fail(DCL_E_ARG, "model is NULL");
  if (!m->loaded) return fail(DCL_E_STATE, "weights not loaded");
  if (!hidden) return fail(DCL_E_ARG, "hidden is NULL");
  if ((reinterpret_cast<uintptr_t>(hidden) & 15) != 0) return fail(DCL_E_ARG, "hidden must be 16-byte aligned");
  if (n < 1 || n > (1 << 22)) return fail(DCL_E_ARG, "n=%d outside [1, 2^22]", n);
  if ((long)n * m->cfg.d_model >= (1L << 31))
    return fail(DCL_E_UNSUPPORTED, "n=%d rows of %d: the LM-head GEMM addresses at most 2^31 elements", n,
                m->cfg.d_model);
  if (!out.top1 || !out.top2 || !out.conf || !out.p2 || !out.lse) return fail(DCL_E_ARG, "an output array is NULL");
  if (!ws) return fail(DCL_E_ARG, "workspace is NULL");
  if ((reinterpret_cast<uintptr_t>(ws) & 255) != 0) return fail(DCL_E_ARG, "workspace must be 256-byte aligned");
  const ScoreLayout L = score_layout(m->cfg, n);
  if (ws_bytes < L.total) return fail(DCL_E_WORKSPACE, "workspace %zu bytes < required %zu", ws_bytes, L.total);
  (void)hipGetLastError();
  int32_t* rows = at<int32_t>(ws, L.rows);
  int32_t* count = at<int32_t>(ws, L.count);
  hipStream_t s = stream;
  launch_iota(rows, count, n, stream);
  LmOut lo;
  lo.pm1 = at<float>(ws, L.pm1);
  lo.pi1 = at<int32_t>(ws, L.pi1);
  lo.pm2 = at<float>(ws, L.pm2);
  lo.pi2 = at<int32_t>(ws, L.pi2);
  lo.ps = at<float>(ws, L.ps);
  lo.pt = at<float>(ws, L.pt);
  lo.n_vt = L.n_vt;
  lo.count = count;
  {
    PROF(P_LM);
    gemm_lmhead(at<bf16_t>(m->wbuf, m->lay.lm), static_cast<const bf16_t*>(hidden), m->cfg.vocab, n, m->cfg.d_model,
                lo, stream);
  }
  {
    PROF(P_MERGE);
    launch_merge(lo.pm1, lo.pi1, lo.pm2, lo.pi2, lo.ps, lo.pt, L.n_vt, rows, count, n, out, stream);
  }
  return hip_check(hipGetLastError(), "score_hidden launch");
}

dcl_status dcl_debug_logits(dcl_model_t model, const int32_t* tokens, int32_t B, int32_t S, const dcl_kv* kv,
                            const int32_t* rows, int32_t n_rows, float* out, void* hidden_out, void* ws,
                            size_t ws_bytes, hipStream_t stream) {
  Model* m = reinterpret_cast<Model*>(model);
  dcl_status st = check_step_args(m, tokens, B, S, kv, ws, ws_bytes);
  if (st != DCL_OK) return st;
  if (!rows || !out) return fail(DCL_E_ARG, "rows / out is NULL");
  if (n_rows < 1 || n_rows > B * S) return fail(DCL_E_ARG, "n_rows %d outside [1, B*S]", n_rows);
  const dcl_config& c = m->cfg;
  const StepLayout L = step_layout(c, B, S, kv ? kv->prefix_len : 0);
  (void)hipGetLastError();
  const int pending = run_forward(m, tokens, B, S, kv, ws, L, stream);
  // the row count goes to the device through a kernel argument (no host buffer to keep alive)
  int32_t* count = at<int32_t>(ws, L.count);
  launch_iota(at<int32_t>(ws, L.pm1), count, n_rows, stream);
  bf16_t* hf = at<bf16_t>(ws, L.hf);
  launch_rmsnorm(at<float>(ws, L.r), at<float>(m->wbuf, m->lay.gf), hf, L.T, c.d_model, c.rms_eps, rows, count,
                 at<float>(ws, L.part), pending, stream);
  gemm_store_f32(at<bf16_t>(m->wbuf, m->lay.lm), hf, c.vocab, n_rows, c.d_model, out, stream);
  if (hidden_out) {
    st = hip_check(hipMemcpyAsync(hidden_out, hf, (size_t)n_rows * c.d_model * 2, hipMemcpyDeviceToDevice, stream),
                   "hipMemcpyAsync(hidden_out)");
    if (st != DCL_OK) return st;
  }
  return hip_check(hipGetLastError(), "debug_logits launch");
}

dcl_status dcl_debug_layer(dcl_model_t model, int32_t B, int32_t S, const dcl_kv* kv, int32_t layer,
                           const float* r_in, dcl_layer_taps taps, void* ws, size_t ws_bytes, hipStream_t stream) {
  Model* m = reinterpret_cast<Model*>(model);
  dcl_status st = check_shape_args(m, B, S, kv);
  if (st != DCL_OK) return st;
  if (layer < 0 || layer >= m->cfg.n_layers) return fail(DCL_E_ARG, "layer %d outside [0, %d)", layer, m->cfg.n_layers);
  if (!r_in) return fail(DCL_E_ARG, "r_in is NULL");
  if (!m->loaded) return fail(DCL_E_STATE, "weights not loaded");
  st = check_workspace(m, B, S, kv ? kv->prefix_len : 0, ws, ws_bytes);
  if (st != DCL_OK) return st;
  const StepLayout L = step_layout(m->cfg, B, S, kv ? kv->prefix_len : 0);
  (void)hipGetLastError();
  st = hip_check(hipMemcpyAsync(at<float>(ws, L.r), r_in, (size_t)B * S * m->cfg.d_model * 4, hipMemcpyDeviceToDevice,
                                stream), "hipMemcpyAsync(r_in)");
  if (st != DCL_OK) return st;
  run_layer(m, layer, B, S, kv, ws, L, stream, 0, false, &taps);
  return hip_check(hipGetLastError(), "debug_layer launch");
}

dcl_status dcl_debug_gemm_plan(int32_t Nw, int32_t T, int32_t K, int32_t lm_head, int32_t max_split, int32_t* info) {
  if (!info) return fail(DCL_E_ARG, "info is NULL");
  if (Nw < 1 || T < 1 || K < 1 || max_split < 1 || max_split > kMaxSplit)
    return fail(DCL_E_ARG, "Nw=%d T=%d K=%d max_split=%d outside their ranges", Nw, T, K, max_split);
  const GemmPlan p = plan_gemm(Nw, T, K, lm_head ? kLmTile : 0, lm_head ? 1 : max_split);
  int shape[6];
  gemm_cfg_shape(p.cfg, shape);
  info[0] = p.cfg;
  info[1] = p.nsplit;
  for (int i = 0; i < 6; ++i) info[2 + i] = shape[i];
  return DCL_OK;
}

dcl_status dcl_profile_enable(int32_t on) {
  if (on != 0 && on != 1) return fail(DCL_E_ARG, "on must be 0 or 1");
  if (on) {
    g_prof.drain(true);
    for (int i = 0; i < DCL_PROF_CLASSES; ++i) {
      g_prof.launches[i] = 0;
      g_prof.ms[i] = 0.0;
    }
  }
  g_prof.on = on != 0;
  return DCL_OK;
}

dcl_status dcl_profile_read(dcl_profile* out) {
  if (!out) return fail(DCL_E_ARG, "out is NULL");
  g_prof.drain(true);
  for (int i = 0; i < DCL_PROF_CLASSES; ++i) {
    out->launches[i] = g_prof.launches[i];
    out->ms[i] = g_prof.ms[i];
  }
  return DCL_OK;
}

}  // extern "C"
