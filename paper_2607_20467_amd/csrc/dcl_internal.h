// Internal declarations of libdcl: device helpers, the model handle, kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "dcl.h"

namespace dcl {

// Raise a kernel's dynamic-LDS limit to `bytes` once per device (devices 0-31): the attribute
// belongs to the device the call is made on, so the first launch on each device sets it and later
// launches only read the mask. Safe when several host threads launch at once.
inline void ensure_dynamic_lds(const void* kern, size_t bytes, std::atomic<uint32_t>& devices_done) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return;
  const uint32_t bit = 1u << (dev & 31);
  if (devices_done.load(std::memory_order_acquire) & bit) return;
  if (hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes) == hipSuccess)
    devices_done.fetch_or(bit, std::memory_order_acq_rel);
}

typedef uint16_t bf16_t;  // bfloat16 bit pattern
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// float -> bfloat16, round to nearest even, by gfx950's v_cvt_pk_bf16_f32. Checked on MI355X
// against the bit-level definition (add 0x7fff + lsb, truncate) for all 2^32 inputs: identical
// for every non-NaN value, denormals and infinities included; NaN stays NaN.
__device__ __forceinline__ bf16_t f2bf(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }
// Two conversions in one instruction: lo in bits 0-15, hi in bits 16-31.
__device__ __forceinline__ uint32_t f2bf2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}
__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// One wave-wide global -> LDS copy of 16 bytes per lane (global_load_lds_dwordx4); lane i lands at
// lds + 16 i, so `lds` must be wave-uniform. Issued from inline assembly with M0 = the LDS
// destination: the compiler then neither counts the copy as outstanding LDS traffic (which makes
// it wait for lgkmcnt(0) before every fragment read) nor inserts vmcnt(0) before LDS reads that
// might alias it. Callers track completion themselves (s_waitcnt vmcnt + barrier).
__device__ __forceinline__ void dma16_at(const void* g, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
               ::"s"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(g) : "memory", "m0");
}
// LDS byte address of a pointer into __shared__ memory (wave-uniform, no null check)
__device__ __forceinline__ uint32_t lds_addr_of(const void* lds) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)lds);
}
__device__ __forceinline__ void dma16(const void* g, const void* lds) { dma16_at(g, lds_addr_of(lds)); }

// Packed-weight layout (byte offsets into the caller's weight buffer).
struct LayerOffsets {
  size_t wqkv, bqkv, wo, wgu, wd, g1, g2;
};
struct WeightLayout {
  size_t embed, gf, lm, rope, total;
  LayerOffsets layer[512];
};

struct Model {
  dcl_config cfg;
  WeightLayout lay;
  void* wbuf = nullptr;  // borrowed
  bool loaded = false;
  int qkv_rows() const { return (cfg.n_heads + 2 * cfg.n_kv_heads) * cfg.head_dim; }
};

// Step workspace layout.
// Fresh keys/values of a step: with a cached prefix of P positions the P mod 8 newest cached keys are
// carried in front of the S fresh ones (koff = P mod 8), so attention reads the cache only in whole
// 8-key chunks [0, P - koff); Sk = koff + S keys per (sequence, kv head), Sp = Sk rounded up to 8.
struct StepLayout {
  size_t r, u, q, k, vt, o, a, rows, count, hf, pm1, pi1, pm2, pi2, ps, pt, part, total;
  int T, S, Sk, Sp, koff, n_vt;
};

// Vocabulary tile of the fused LM-head reduction (vocab ids per partial) and the number of waves
// that split it (their partials merge through LDS in the GEMM epilogue).
constexpr int kLmTile = 128;
constexpr int kLmWaves = 2;

// ---------------------------------------------------------------- launchers (stream-ordered)
void launch_embed(const int32_t* tokens, const bf16_t* E, float* r, int T, int d, int V, hipStream_t s);
// u = bf16(rmsnorm(r) * g). With nP > 0, first r + P[0] + ... + P[nP-1] (slices [T, d]) in that
// order, written back to r unless `rows` selects the rows (final norm).
void launch_rmsnorm(float* r, const float* g, bf16_t* u, int T, int d, float eps, const int32_t* rows,
                    const int32_t* count, const float* P, int nP, hipStream_t s);
void launch_compact(const int32_t* tokens, const int32_t* p, int B, int S, int gen_end, int mask_id,
                    int score_all, int32_t* rows, int32_t* count, dcl_row_stats st, hipStream_t s);
void launch_merge(const float* pm1, const int32_t* pi1, const float* pm2, const int32_t* pi2,
                  const float* ps, const float* pt, int n_vt, const int32_t* rows, const int32_t* count,
                  int max_rows, dcl_row_stats st, hipStream_t s);
void launch_iota(int32_t* rows, int32_t* count, int n, hipStream_t s);
// block_len > 0: semi-AR blocks of block_len positions from block_origin; the window and the re-mask
// stop at the end of the block holding p.
void launch_select(int32_t* tokens, int B, int S, int32_t* p, int gen_end, int L, int block_origin, int block_len,
                   float tau_c, float tau_d, int mask_id, dcl_row_stats st, int32_t* k_raw, int32_t* k_eff,
                   uint32_t flags, hipStream_t s, int32_t* k_hist = nullptr);
void launch_remask(int32_t* tokens, int B, int S, const int32_t* p, int gen_end, int L, int block_origin,
                   int block_len, int mask_id, hipStream_t s);
void launch_pack_rows(const void* src, int src_dtype, bf16_t* dst, int rows, int cols, int mode,
                      int dh, int dst_row0, hipStream_t s);
void launch_pack_vec(const void* src, int src_dtype, float* dst, int n, int mode, int dh, int dst0,
                     hipStream_t s);

// GEMM family: C[w, t] = sum_k W[w, k] X[t, k], W bf16 [Nw, K], X bf16 [T, K] (both K-contiguous).
struct QkvOut {
  bf16_t *q, *k, *vt;
  const float* bias;     // packed order, or null
  const float2* rope;    // [max_pos, dh/2] (cos, sin) or null (RoPE off)
  int H, Hkv, dh, S, Sp, pos0;
  int Sk = 0, koff = 0;  // fresh key rows per (b, kv head) and the slot of token 0 (0, 0: Sk = S)
};
struct LmOut {
  float *pm1, *pm2, *ps;
  float* pt;  // sum exp(l - m1) * (l - m1) per partial (entropy), relative like ps
  int32_t *pi1, *pi2;
  int n_vt;
  const int32_t* count;  // number of valid X rows (device)
  int exclude = -1;      // vocabulary id left out of the reduction (mask suppression), -1: none
};
// Tile shape / split-K choice for one GEMM shape (host).
struct GemmPlan {
  int cfg, nsplit, tiles;
};
// force_bw: restrict to tiles of that many weight rows (0: any); max_split: largest K-split factor.
GemmPlan plan_gemm(int Nw, int T, int K, int force_bw, int max_split);
// Tile of configuration `cfg`: {weight rows, tokens, K depth per stage, stages, waves along W, waves along T}.
void gemm_cfg_shape(int cfg, int* shape);
constexpr int kMaxSplit = 4;  // K-split slices of the residual GEMMs
void gemm_qkv(const bf16_t* W, const bf16_t* X, int Nw, int T, int K, const QkvOut& o, hipStream_t s);
// r += W X^T, either in place (returns 0) or as n float32 slices P[s][T][Nw] that the next RMSNorm
// folds into r in split order (returns n > 1). P may be null (in place only).
int gemm_resid(const bf16_t* W, const bf16_t* X, int Nw, int T, int K, float* r, float* P, hipStream_t s);
void gemm_swiglu(const bf16_t* W, const bf16_t* X, int Nw, int T, int K, bf16_t* a, hipStream_t s);
void gemm_lmhead(const bf16_t* W, const bf16_t* X, int V, int T, int K, const LmOut& o, hipStream_t s);
void gemm_store_f32(const bf16_t* W, const bf16_t* X, int Nw, int T, int K, float* out, hipStream_t s);

// Non-causal attention over [cache (P keys) || fresh (S keys)].
struct AttnArgs {
  const bf16_t *q, *k, *vt;      // [B,H,S,dh] queries; [B,Hkv,Sk,dh], [B,Hkv,dh,Sp] fresh keys / values
  const bf16_t *kc, *vc;         // [B,Hkv,Pc,dh], [B,Hkv,dh,Pc] (first P positions used) or null
  bf16_t* o;                     // [B,S,H*dh]
  int B, H, Hkv, dh, S, Sp, P, Pc;
  float scale_log2;              // log2(e) / sqrt(dh)
  int Sk = 0;                    // keys per (b, kv head) in k / vt; 0: Sk = S. P (the keys read from the
                                 // cache) must be a multiple of 8: the P mod 8 newest cached keys of a
                                 // ragged prefix are carried into the front of k / vt (Sk = P mod 8 + S)
};
void launch_attention(const AttnArgs& a, hipStream_t s);
// The koff = P mod 8 newest cached keys [P - koff, P) and their values into slots [0, koff) of the fresh
// buffers k [B,Hkv,Sk,dh] and vt [B,Hkv,dh,Sp] (cache kc [B,Hkv,Pc,dh], vc [B,Hkv,dh,Pc]).
void launch_kv_carry(const bf16_t* kc, const bf16_t* vc, bf16_t* k, bf16_t* vt, int B, int Hkv, int Sk, int Sp,
                     int dh, int P, int Pc, hipStream_t s);
// Fresh keys k [B,Hkv,Sk,dh] and values vt [B,Hkv,dh,Sp] of tokens 0..S-1 (slots koff + s) into a cache at
// positions [P, P + S) (kc [B,Hkv,Pc,dh], vc [B,Hkv,dh,Pc]).
void launch_kv_writeback(const bf16_t* k, const bf16_t* vt, bf16_t* kc, bf16_t* vc, int B, int Hkv, int S, int Sk,
                         int Sp, int koff, int dh, int P, int Pc, hipStream_t s);

}  // namespace dcl
