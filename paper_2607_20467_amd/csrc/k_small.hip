// Memory-bound kernels of the denoising step: embedding gather, RMSNorm, scored-row compaction,
// merge of the fused LM-head partials, DCV + draft selection, weight packing.
#include <float.h>
#include <limits.h>

#include "dcl_internal.h"

namespace dcl {

// ---------------------------------------------------------------- embedding gather
// r[t, :] = E[tokens[t], :] widened to float32; ids outside [0, V) give a zero row.
__global__ void __launch_bounds__(256) embed_kernel(const int32_t* __restrict__ tokens,
                                                   const bf16_t* __restrict__ E, float* __restrict__ r,
                                                   int T, int d, int V) {
  const int chunks = d / 8;
  long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)T * chunks) return;
  int t = (int)(idx / chunks), c = (int)(idx % chunks);
  int id = tokens[t];
  float4 lo = {0.f, 0.f, 0.f, 0.f}, hi = lo;
  if (id >= 0 && id < V) {
    uint4 v = *reinterpret_cast<const uint4*>(E + (size_t)id * d + c * 8);
    lo = {__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xFFFF0000u),
          __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xFFFF0000u)};
    hi = {__uint_as_float(v.z << 16), __uint_as_float(v.z & 0xFFFF0000u),
          __uint_as_float(v.w << 16), __uint_as_float(v.w & 0xFFFF0000u)};
  }
  float4* dst = reinterpret_cast<float4*>(r + (size_t)t * d + c * 8);
  dst[0] = lo;
  dst[1] = hi;
}

void launch_embed(const int32_t* tokens, const bf16_t* E, float* r, int T, int d, int V, hipStream_t s) {
  long n = (long)T * (d / 8);
  if (n == 0) return;
  hipLaunchKernelGGL(embed_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, tokens, E, r, T, d, V);
}

// ---------------------------------------------------------------- RMSNorm
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// One 256-thread workgroup per row: u = bf16(r * rsqrt(mean(r^2) + eps) * g). Each thread holds
// NV float4 of the row in registers (all loads issued at once), the sum of squares is reduced
// across the workgroup in a fixed order. With `rows`, output row j normalises input row rows[j]
// (j < *count); otherwise output row j = input row j. T is the number of rows of r.
// With nP > 0 the row first takes the K-split slices of the residual GEMM that produced it:
// r + P[0] + ... + P[nP-1] (each [T, d], added in that order); without `rows` the sum is written
// back to r (with `rows`, the final norm, r is not needed afterwards and stays as it is).
template <int NV, int NP>
__global__ void __launch_bounds__(256) rmsnorm_kernel(float* __restrict__ r, const float* __restrict__ g,
                                                     bf16_t* __restrict__ u, int T, int d, float eps,
                                                     const int32_t* __restrict__ rows,
                                                     const int32_t* __restrict__ count,
                                                     const float* __restrict__ P) {
  __shared__ float red[4];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int j = blockIdx.x;
  const int n = rows ? *count : T;
  if (j >= n) return;
  const int src = rows ? rows[j] : j;
  bf16_t* y = u + (size_t)j * d;
  const int d4 = d >> 2;
  if (src < 0 || src >= T) {  // row index outside the residual buffer: zero row
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int c = tid + v * 256;
      if (c < d4) *reinterpret_cast<uint2*>(y + 4 * c) = make_uint2(0, 0);
    }
    return;
  }
  float4* x = reinterpret_cast<float4*>(r + (size_t)src * d);
  const float4* g4 = reinterpret_cast<const float4*>(g);
  float4 v[NV], gv[NV];  // the gains are loaded with the row, not after the reduction
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int c = tid + k * 256;
    v[k] = c < d4 ? x[c] : make_float4(0.f, 0.f, 0.f, 0.f);
    gv[k] = c < d4 ? g4[c] : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  if (NP > 0) {
    // every slice load is issued before the first add (one memory round trip, not NP); the adds
    // then run in split order, so the sum is the same bit pattern as a sequential fold
    float4 q[NP > 0 ? NP : 1][NV];
#pragma unroll
    for (int sp = 0; sp < NP; ++sp) {
      const float4* ps = reinterpret_cast<const float4*>(P + ((size_t)sp * T + src) * d);
#pragma unroll
      for (int k = 0; k < NV; ++k) {
        const int c = tid + k * 256;
        q[sp][k] = c < d4 ? ps[c] : make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
#pragma unroll
    for (int sp = 0; sp < NP; ++sp)
#pragma unroll
      for (int k = 0; k < NV; ++k) {
        v[k].x += q[sp][k].x; v[k].y += q[sp][k].y; v[k].z += q[sp][k].z; v[k].w += q[sp][k].w;
      }
    if (!rows) {
#pragma unroll
      for (int k = 0; k < NV; ++k) {
        const int c = tid + k * 256;
        if (c < d4) x[c] = v[k];
      }
    }
  }
#pragma unroll
  for (int k = 0; k < NV; ++k) ss += v[k].x * v[k].x + v[k].y * v[k].y + v[k].z * v[k].z + v[k].w * v[k].w;
  ss = wave_sum(ss);
  if (lane == 0) red[wid] = ss;
  __syncthreads();
  const float tot = (red[0] + red[1]) + (red[2] + red[3]);
  const float inv = 1.0f / sqrtf(tot / (float)d + eps);
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int c = tid + k * 256;
    if (c < d4) {
      const float4 w = gv[k];
      uint2 o;
      o.x = f2bf2(v[k].x * inv * w.x, v[k].y * inv * w.y);
      o.y = f2bf2(v[k].z * inv * w.z, v[k].w * inv * w.w);
      *reinterpret_cast<uint2*>(y + 4 * c) = o;
    }
  }
}

template <int NV>
static void launch_rmsnorm_nv(float* r, const float* g, bf16_t* u, int T, int d, float eps, const int32_t* rows,
                              const int32_t* count, const float* P, int nP, hipStream_t s) {
  switch (nP) {
    case 0: hipLaunchKernelGGL((rmsnorm_kernel<NV, 0>), dim3(T), dim3(256), 0, s, r, g, u, T, d, eps, rows, count, P); break;
    case 1: hipLaunchKernelGGL((rmsnorm_kernel<NV, 1>), dim3(T), dim3(256), 0, s, r, g, u, T, d, eps, rows, count, P); break;
    case 2: hipLaunchKernelGGL((rmsnorm_kernel<NV, 2>), dim3(T), dim3(256), 0, s, r, g, u, T, d, eps, rows, count, P); break;
    case 3: hipLaunchKernelGGL((rmsnorm_kernel<NV, 3>), dim3(T), dim3(256), 0, s, r, g, u, T, d, eps, rows, count, P); break;
    default: hipLaunchKernelGGL((rmsnorm_kernel<NV, 4>), dim3(T), dim3(256), 0, s, r, g, u, T, d, eps, rows, count, P); break;
  }
}

void launch_rmsnorm(float* r, const float* g, bf16_t* u, int T, int d, float eps, const int32_t* rows,
                    const int32_t* count, const float* P, int nP, hipStream_t s) {
  if (T == 0) return;
  static_assert(kMaxSplit <= 4, "rmsnorm folds at most four split-K slices");
  const int nv = (d / 4 + 255) / 256;
  if (nv <= 1) launch_rmsnorm_nv<1>(r, g, u, T, d, eps, rows, count, P, nP, s);
  else if (nv <= 2) launch_rmsnorm_nv<2>(r, g, u, T, d, eps, rows, count, P, nP, s);
  else if (nv <= 4) launch_rmsnorm_nv<4>(r, g, u, T, d, eps, rows, count, P, nP, s);
  else launch_rmsnorm_nv<8>(r, g, u, T, d, eps, rows, count, P, nP, s);
}

// ---------------------------------------------------------------- scored-row compaction
// Single workgroup: rows = flat indices b*S+i of scored positions in increasing order, count = R.
// Unscored positions get the sentinel statistics.
__global__ void __launch_bounds__(1024) compact_kernel(const int32_t* __restrict__ tokens,
                                                      const int32_t* __restrict__ p, int B, int S,
                                                      int gen_end, int mask_id, int score_all,
                                                      int32_t* __restrict__ rows, int32_t* __restrict__ count,
                                                      dcl_row_stats st) {
  __shared__ int wave_tot[16];
  __shared__ int base;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  if (tid == 0) base = 0;
  __syncthreads();
  const int total = B * S;
  for (int start = 0; start < total; start += 1024) {
    int idx = start + tid;
    int flag = 0;
    if (idx < total) {
      int b = idx / S, i = idx % S;
      flag = (i >= p[b] && i < gen_end && (score_all || tokens[idx] == mask_id)) ? 1 : 0;
      if (!flag) {
        st.top1[idx] = -1;
        st.top2[idx] = -1;
        st.conf[idx] = -1.f;
        st.p2[idx] = -1.f;
        st.lse[idx] = 0.f;
        if (st.entropy) st.entropy[idx] = -1.f;
      }
    }
    unsigned long long m = __ballot(flag);
    int before = __popcll(m & ((1ull << lane) - 1ull));
    if (lane == 0) wave_tot[wid] = __popcll(m);
    __syncthreads();
    int off = base;
    for (int w = 0; w < wid; ++w) off += wave_tot[w];
    if (flag) rows[off + before] = idx;
    __syncthreads();
    if (tid == 0) {
      int add = 0;
      for (int w = 0; w < 16; ++w) add += wave_tot[w];
      base += add;
    }
    __syncthreads();
  }
  if (tid == 0) *count = base;
}

void launch_compact(const int32_t* tokens, const int32_t* p, int B, int S, int gen_end, int mask_id,
                    int score_all, int32_t* rows, int32_t* count, dcl_row_stats st, hipStream_t s) {
  hipLaunchKernelGGL(compact_kernel, dim3(1), dim3(1024), 0, s, tokens, p, B, S, gen_end, mask_id, score_all,
                     rows, count, st);
}

// ---------------------------------------------------------------- top-2 / sum-exp merge
struct Top2 {
  float m1, m2;
  int i1, i2;
};
// (value desc, id asc) ordering
__device__ __forceinline__ bool better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}
__device__ __forceinline__ Top2 top2_merge(Top2 a, Top2 b) {
  Top2 o;
  if (better(a.m1, a.i1, b.m1, b.i1)) {
    o.m1 = a.m1; o.i1 = a.i1;
    if (better(a.m2, a.i2, b.m1, b.i1)) { o.m2 = a.m2; o.i2 = a.i2; } else { o.m2 = b.m1; o.i2 = b.i1; }
  } else {
    o.m1 = b.m1; o.i1 = b.i1;
    if (better(b.m2, b.i2, a.m1, a.i1)) { o.m2 = b.m2; o.i2 = b.i2; } else { o.m2 = a.m1; o.i2 = a.i1; }
  }
  return o;
}

// Running (top-2, S, Tm) of a set of vocabulary tiles; S = sum exp(l - m1) and
// Tm = sum exp(l - m1) (l - m1) are relative to the set's own top-1 value m1.
struct RowAcc {
  Top2 t;
  float s, tm;
};
// Union of two disjoint sets: the relative sums move to the new top-1 value M (a term
// exp(l - m) (l - m) becomes exp(l - M) (l - M) = e^(m-M) (exp(l - m) (l - m) + exp(l - m) (m - M))).
// Symmetric in its arguments (distinct ids, commutative float adds), so every lane of a butterfly
// computes the same bits.
__device__ __forceinline__ RowAcc row_merge(const RowAcc& a, const RowAcc& b) {
  RowAcc o;
  o.t = top2_merge(a.t, b.t);
  const float M = o.t.m1;
  const bool ea_ok = a.t.m1 != -INFINITY, eb_ok = b.t.m1 != -INFINITY;
  const float da = ea_ok ? a.t.m1 - M : 0.f, db = eb_ok ? b.t.m1 - M : 0.f;
  const float ea = ea_ok ? __expf(da) : 0.f, eb = eb_ok ? __expf(db) : 0.f;
  o.s = a.s * ea + b.s * eb;
  o.tm = ea * (a.tm + a.s * da) + eb * (b.tm + b.s * db);
  return o;
}

// One wavefront per scored row folds the row's per-vocabulary-tile partials in a fixed order:
// lane l takes tiles l, l + 64, ... (four loads in flight per lane), then a fixed butterfly. The
// result is bitwise reproducible. With M = the row maximum and S = sum_v exp(l_v - M):
// conf = 1 / S, p2 = exp(m2 - M) / S, lse = M + log S, entropy = log S - Tm / S.
__global__ void __launch_bounds__(256) merge_kernel(const float* __restrict__ pm1, const int32_t* __restrict__ pi1,
                                                   const float* __restrict__ pm2, const int32_t* __restrict__ pi2,
                                                   const float* __restrict__ ps, const float* __restrict__ pt,
                                                   int n_vt, const int32_t* __restrict__ rows,
                                                   const int32_t* __restrict__ count, dcl_row_stats st) {
  const int lane = threadIdx.x & 63;
  const int j = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (j >= *count) return;
  const size_t base = (size_t)j * n_vt;
  RowAcc acc = {{-INFINITY, -INFINITY, INT_MAX, INT_MAX}, 0.f, 0.f};
  constexpr int U = 4;
  for (int v0 = lane; v0 < n_vt; v0 += 64 * U) {
    RowAcc x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = v0 + 64 * u;
      if (v < n_vt) {
        x[u].t = {pm1[base + v], pm2[base + v], pi1[base + v], pi2[base + v]};
        x[u].s = ps[base + v];
        x[u].tm = pt[base + v];
      } else {
        x[u] = {{-INFINITY, -INFINITY, INT_MAX, INT_MAX}, 0.f, 0.f};
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) acc = row_merge(acc, x[u]);
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    RowAcc x;
    x.t = {__shfl_xor(acc.t.m1, o, 64), __shfl_xor(acc.t.m2, o, 64), __shfl_xor(acc.t.i1, o, 64),
           __shfl_xor(acc.t.i2, o, 64)};
    x.s = __shfl_xor(acc.s, o, 64);
    x.tm = __shfl_xor(acc.tm, o, 64);
    acc = row_merge(acc, x);
  }
  if (lane == 0) {
    const int row = rows[j];
    const float s = acc.s;
    st.top1[row] = acc.t.i1;
    st.top2[row] = acc.t.i2;
    st.conf[row] = 1.0f / s;
    st.p2[row] = __expf(acc.t.m2 - acc.t.m1) / s;
    st.lse[row] = acc.t.m1 + logf(s);
    if (st.entropy) st.entropy[row] = logf(s) - acc.tm / s;
  }
}

void launch_merge(const float* pm1, const int32_t* pi1, const float* pm2, const int32_t* pi2, const float* ps,
                  const float* pt, int n_vt, const int32_t* rows, const int32_t* count, int max_rows,
                  dcl_row_stats st, hipStream_t s) {
  if (max_rows == 0) return;
  hipLaunchKernelGGL(merge_kernel, dim3((max_rows + 3) / 4), dim3(256), 0, s, pm1, pi1, pm2, pi2, ps, pt, n_vt, rows,
                     count, st);
}

// rows[j] = j for j < n, count = n (row map of dcl_score_hidden and dcl_debug_logits' copy).
__global__ void iota_kernel(int32_t* __restrict__ rows, int32_t* __restrict__ count, int n) {
  int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j < n) rows[j] = j;
  if (j == 0) *count = n;
}

void launch_iota(int32_t* rows, int32_t* count, int n, hipStream_t s) {
  hipLaunchKernelGGL(iota_kernel, dim3((n + 255) / 256), dim3(256), 0, s, rows, count, n);
}

// ---------------------------------------------------------------- DCV + drafts + remask
// End of the window for a pointer at `pos`: gen_end, or with semi-AR blocks (block_len > 0, blocks of
// block_len positions tiling the line from block_origin) the end of the block holding pos, if earlier.
__device__ __forceinline__ int window_end(int pos, int gen_end, int block_origin, int block_len) {
  if (block_len <= 0) return gen_end;
  const long d = (long)pos - block_origin;
  const long q = d >= 0 ? d / block_len : -((-d + block_len - 1) / block_len);  // floor(d / block_len)
  return (int)min((long)gen_end, (long)block_origin + (long)block_len * (q + 1));
}

// One workgroup per sequence.
__global__ void __launch_bounds__(256) select_kernel(int32_t* __restrict__ tokens, int S, int32_t* __restrict__ p,
                                                    int gen_end, int L, int block_origin, int block_len, float tau_c,
                                                    float tau_d, int mask_id, dcl_row_stats st,
                                                    int32_t* __restrict__ k_raw, int32_t* __restrict__ k_eff,
                                                    uint32_t flags, int32_t* __restrict__ k_hist) {
  __shared__ int red[4];
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  int32_t* x = tokens + (size_t)b * S;
  const int32_t* top1 = st.top1 + (size_t)b * S;
  const float* cf = st.conf + (size_t)b * S;
  const float* p2 = st.p2 + (size_t)b * S;
  const bool margin = (flags & DCL_SEL_MARGIN) != 0;
  // the acceptance statistic: the confidence, or the top-1/top-2 margin (unscored rows stay -1)
  auto conf_at = [&](int j) -> float { return (margin && cf[j] >= 0.f) ? cf[j] - p2[j] : cf[j]; };
  const int pb = p[b];
  if (pb < 0 || pb >= gen_end) {  // finished (or invalid) pointer: the sequence is left untouched
    if (tid == 0) {
      if (k_raw) k_raw[b] = 0;
      if (k_eff) k_eff[b] = 0;
    }
    return;
  }
  const int L_eff = min(L, window_end(pb, gen_end, block_origin, block_len) - pb);
  // window ends computed in 64-bit: p + L may exceed INT_MAX for a huge L
  const int draft_start = (int)min((long)pb + L, (long)gen_end);
  if (flags & DCL_SEL_NONCONTIGUOUS) {
    // Eq. threshold_pd in the window: independent commits of every masked, scored row above tau_c
    __shared__ int npass[4];
    __shared__ unsigned long long bestk[4];
    int n = 0;
    unsigned long long best = 0;  // (conf bits, ~j): max picks the highest conf, then the lowest j
    for (int j = pb + tid; j < pb + L_eff; j += 256) {
      if (x[j] == mask_id && top1[j] >= 0) {
        const float c = conf_at(j);
        if (c > tau_c) {
          x[j] = top1[j];
          ++n;
        }
        const unsigned long long k = ((unsigned long long)__float_as_uint(fmaxf(c, 0.f)) << 32) |
                                     (unsigned long long)(0xFFFFFFFFu - (uint32_t)j);
        best = k > best ? k : best;
      }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      n += __shfl_xor(n, o, 64);
      const unsigned long long v = __shfl_xor(best, o, 64);
      best = v > best ? v : best;
    }
    if (lane == 0) {
      npass[wid] = n;
      bestk[wid] = best;
    }
    __syncthreads();
    const int passing = (npass[0] + npass[1]) + (npass[2] + npass[3]);
    unsigned long long bk = bestk[0];
    for (int w = 1; w < 4; ++w) bk = bestk[w] > bk ? bestk[w] : bk;
    int Ke = passing;
    if (passing == 0 && bk != 0 && !(flags & DCL_SEL_NO_PROGRESS_GUARD)) {
      const int jb = (int)(0xFFFFFFFFu - (uint32_t)(bk & 0xFFFFFFFFull));
      if (tid == 0) x[jb] = top1[jb];
      Ke = 1;
    }
    __syncthreads();
    // p <- first position >= p still masked (the verified prefix ends there)
    int firstm = gen_end;
    for (int j = pb + tid; j < gen_end; j += 256)
      if (x[j] == mask_id) {
        firstm = j;
        break;
      }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) firstm = min(firstm, __shfl_xor(firstm, o, 64));
    __syncthreads();
    if (lane == 0) npass[wid] = firstm;
    __syncthreads();
    if (tid == 0) {
      p[b] = min(min(npass[0], npass[1]), min(npass[2], npass[3]));
      if (k_raw) k_raw[b] = passing;
      if (k_eff) k_eff[b] = Ke;
      if (k_hist) atomicAdd(&k_hist[Ke], 1);  // Ke <= L_eff <= L
    }
    return;
  }
  // K = index of the first window row that fails conf > tau_c (Eq. compute_k), L_eff if none.
  int first = L_eff;
  for (int j = tid; j < L_eff; j += 256)
    if (!(conf_at(pb + j) > tau_c)) first = min(first, j);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) first = min(first, __shfl_xor(first, o, 64));
  if (lane == 0) red[wid] = first;
  __syncthreads();
  const int K = min(min(red[0], red[1]), min(red[2], red[3]));
  int Ke = K;
  if (!(flags & DCL_SEL_NO_PROGRESS_GUARD) && Ke == 0 && top1[pb] >= 0) Ke = 1;
  for (int j = tid; j < Ke; j += 256) x[pb + j] = top1[pb + j];
  const bool any = (flags & DCL_SEL_SCORE_ALL) != 0;
  int chain_end = gen_end;  // Appendix E: the draft chain ends at the first eligible row that fails
  if (flags & DCL_SEL_CONTIGUOUS_DRAFTS) {
    for (int j = draft_start + tid; j < gen_end; j += 256)
      if ((any || x[j] == mask_id) && !(conf_at(j) > tau_d && top1[j] >= 0)) {
        chain_end = j;
        break;
      }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) chain_end = min(chain_end, __shfl_xor(chain_end, o, 64));
    __syncthreads();  // red[] is free again
    if (lane == 0) red[wid] = chain_end;
    __syncthreads();
    chain_end = min(min(red[0], red[1]), min(red[2], red[3]));
  }
  for (int j = draft_start + tid; j < chain_end; j += 256)
    if ((any || x[j] == mask_id) && conf_at(j) > tau_d && top1[j] >= 0) x[j] = top1[j];
  __syncthreads();
  const int pn = pb + Ke;
  const int stop = (int)min((long)pn + L, (long)window_end(pn, gen_end, block_origin, block_len));
  for (int j = pn + tid; j < stop; j += 256) x[j] = mask_id;
  if (tid == 0) {
    p[b] = pn;
    if (k_raw) k_raw[b] = K;
    if (k_eff) k_eff[b] = Ke;
    if (k_hist) atomicAdd(&k_hist[Ke], 1);  // Ke <= L_eff <= L: histogram of [L + 1] bins
  }
}

// Step (i) alone (Eq. remasking): x[b, p_b : min(p_b + L, gen_end)) = mask_id for every sequence
// with 0 <= p_b < gen_end; one workgroup per sequence.
__global__ void __launch_bounds__(256) remask_kernel(int32_t* __restrict__ tokens, int S,
                                                    const int32_t* __restrict__ p, int gen_end, int L,
                                                    int block_origin, int block_len, int mask_id) {
  const int b = blockIdx.x;
  const int pb = p[b];
  if (pb < 0 || pb >= gen_end) return;
  const int stop = (int)min((long)pb + L, (long)window_end(pb, gen_end, block_origin, block_len));
  for (int j = pb + (int)threadIdx.x; j < stop; j += 256) tokens[(size_t)b * S + j] = mask_id;
}

void launch_select(int32_t* tokens, int B, int S, int32_t* p, int gen_end, int L, int block_origin, int block_len,
                   float tau_c, float tau_d, int mask_id, dcl_row_stats st, int32_t* k_raw, int32_t* k_eff,
                   uint32_t flags, hipStream_t s, int32_t* k_hist) {
  hipLaunchKernelGGL(select_kernel, dim3(B), dim3(256), 0, s, tokens, S, p, gen_end, L, block_origin, block_len,
                     tau_c, tau_d, mask_id, st, k_raw, k_eff, flags, k_hist);
}
void launch_remask(int32_t* tokens, int B, int S, const int32_t* p, int gen_end, int L, int block_origin,
                   int block_len, int mask_id, hipStream_t s) {
  hipLaunchKernelGGL(remask_kernel, dim3(B), dim3(256), 0, s, tokens, S, p, gen_end, L, block_origin, block_len,
                     mask_id);
}

// ---------------------------------------------------------------- weight packing (load time)
// Row permutations of the packed layout:
//   mode 0: identity;
//   mode 1: RoPE pair interleave within each head of `dh` rows: source row j (j < dh/2) -> 2j,
//           source row j + dh/2 -> 2j + 1, so a rotation pair sits in adjacent rows;
//   mode 2: gate row f -> 2f;  mode 3: up row f -> 2f + 1 (SwiGLU pairs adjacent).
__device__ __forceinline__ int packed_row(int src, int mode, int dh) {
  if (mode == 1) {
    int h = src / dh, j = src % dh, half = dh / 2;
    return h * dh + (j < half ? 2 * j : 2 * (j - half) + 1);
  }
  if (mode == 2) return 2 * src;
  if (mode == 3) return 2 * src + 1;
  return src;
}

__device__ __forceinline__ float load_src(const void* src, int dtype, size_t i) {
  return dtype == DCL_DTYPE_F32 ? reinterpret_cast<const float*>(src)[i]
                                : bf2f(reinterpret_cast<const bf16_t*>(src)[i]);
}

__global__ void pack_rows_kernel(const void* __restrict__ src, int dtype, bf16_t* __restrict__ dst, int rows,
                                 int cols, int mode, int dh, int dst_row0) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  size_t n = (size_t)rows * cols;
  if (i >= n) return;
  int r = (int)(i / cols), c = (int)(i % cols);
  int pr = dst_row0 + packed_row(r, mode, dh);
  dst[(size_t)pr * cols + c] = f2bf(load_src(src, dtype, i));
}

void launch_pack_rows(const void* src, int src_dtype, bf16_t* dst, int rows, int cols, int mode, int dh,
                      int dst_row0, hipStream_t s) {
  size_t n = (size_t)rows * cols;
  if (n == 0) return;
  hipLaunchKernelGGL(pack_rows_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, src, src_dtype, dst,
                     rows, cols, mode, dh, dst_row0);
}

__global__ void pack_vec_kernel(const void* __restrict__ src, int dtype, float* __restrict__ dst, int n, int mode,
                                int dh, int dst0) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  dst[dst0 + packed_row(i, mode, dh)] = src ? load_src(src, dtype, i) : 0.f;
}

void launch_pack_vec(const void* src, int src_dtype, float* dst, int n, int mode, int dh, int dst0,
                     hipStream_t s) {
  if (n == 0) return;
  hipLaunchKernelGGL(pack_vec_kernel, dim3((n + 255) / 256), dim3(256), 0, s, src, src_dtype, dst, n, mode, dh,
                     dst0);
}

}  // namespace dcl
