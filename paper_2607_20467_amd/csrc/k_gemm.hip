// MFMA bf16 GEMM family for gfx950 with fused epilogues.
//
//   C[w, t] = sum_k W[w, k] * X[t, k]      W: bf16 [Nw, K] (weights, nn.Linear layout)
//                                           X: bf16 [T, K]  (activations, one row per token)
// Both operands are K-contiguous, so every MFMA fragment is one 16-byte load. Weights play the
// MFMA "A" role: a lane of a 16x16 accumulator tile then holds four consecutive weight rows of one
// token, which makes the fused epilogues local to a lane:
//   QKV    + bias, rotate-half RoPE (rotation pairs were interleaved into adjacent rows at load),
//          scattered to q [B,H,S,dh], k [B,Hkv,S,dh] and key-contiguous v [B,Hkv,dh,Sp];
//   RESID  r[t, w] += C (float32 residual stream);
//   SWIGLU a[t, f] = bf16(silu(gate) * up) (gate/up rows interleaved at load);
//   LMHEAD per (token, 128-id vocabulary tile): top-1, top-2 and sum exp(l - top1) — logits stay
//          in registers and never reach memory;
//   F32    plain float32 store (debug logits).
// Tiles: BW weight rows x BT tokens per workgroup, K staged through LDS in steps of 64 with a
// register prefetch of the next step and double-buffered LDS. The block -> tile map is XCD-aware:
// consecutive tiles (which share a weight tile) land on the same XCD and its L2.
#include <float.h>
#include <limits.h>

#include "dcl_internal.h"

namespace dcl {

constexpr int BK = 64;        // K elements per LDS stage
constexpr int LDSP = BK + 8;  // padded LDS row (144 bytes): conflict-free 16-byte fragment reads

__device__ __forceinline__ f32x4_t mfma16(const bf16x8_t& a, const bf16x8_t& b, const f32x4_t& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// ---------------------------------------------------------------- epilogues
// apply(): acc[i][j] holds C[wb + 16 i + 4 (lane/16) + r][tb + 16 j + lane%16], r = 0..3.

struct EpiResid {
  float* r;
  template <int SW, int ST>
  __device__ void apply(f32x4_t (&acc)[SW][ST], int wb, int tb, int lane, int Nw, int T, int) const {
    const int wq = wb + 4 * (lane >> 4), tl = tb + (lane & 15);
#pragma unroll
    for (int j = 0; j < ST; ++j) {
      const int t = tl + 16 * j;
      if (t >= T) continue;
#pragma unroll
      for (int i = 0; i < SW; ++i) {
        const int w = wq + 16 * i;
        if (w >= Nw) continue;
        float4* p = reinterpret_cast<float4*>(r + (size_t)t * Nw + w);
        float4 v = *p;
        v.x += acc[i][j][0]; v.y += acc[i][j][1]; v.z += acc[i][j][2]; v.w += acc[i][j][3];
        *p = v;
      }
    }
  }
};

struct EpiSwiglu {
  bf16_t* a;  // [T, Nw/2]
  template <int SW, int ST>
  __device__ void apply(f32x4_t (&acc)[SW][ST], int wb, int tb, int lane, int Nw, int T, int) const {
    const int F = Nw >> 1;
    const int wq = wb + 4 * (lane >> 4), tl = tb + (lane & 15);
#pragma unroll
    for (int j = 0; j < ST; ++j) {
      const int t = tl + 16 * j;
      if (t >= T) continue;
#pragma unroll
      for (int i = 0; i < SW; ++i) {
        const int w = wq + 16 * i;
        if (w >= Nw) continue;
        const float g0 = acc[i][j][0], u0 = acc[i][j][1], g1 = acc[i][j][2], u1 = acc[i][j][3];
        const float h0 = g0 / (1.0f + __expf(-g0)) * u0;
        const float h1 = g1 / (1.0f + __expf(-g1)) * u1;
        *reinterpret_cast<uint32_t*>(a + (size_t)t * F + (w >> 1)) = (uint32_t)f2bf(h0) | ((uint32_t)f2bf(h1) << 16);
      }
    }
  }
};

struct EpiQkv {
  QkvOut o;
  template <int SW, int ST>
  __device__ void apply(f32x4_t (&acc)[SW][ST], int wb, int tb, int lane, int Nw, int T, int) const {
    const int dh = o.dh, half = dh >> 1;
    const int qrows = o.H * dh, krows = o.Hkv * dh;
    const int wq = wb + 4 * (lane >> 4), tl = tb + (lane & 15);
#pragma unroll
    for (int j = 0; j < ST; ++j) {
      const int t = tl + 16 * j;
      if (t >= T) continue;
      const int b = t / o.S, s = t - b * o.S;
      const int pos = o.pos0 + s;
#pragma unroll
      for (int i = 0; i < SW; ++i) {
        const int w = wq + 16 * i;
        if (w >= Nw) continue;
        float v0 = acc[i][j][0], v1 = acc[i][j][1], v2 = acc[i][j][2], v3 = acc[i][j][3];
        if (o.bias) {
          v0 += o.bias[w]; v1 += o.bias[w + 1]; v2 += o.bias[w + 2]; v3 += o.bias[w + 3];
        }
        if (w < qrows + krows) {
          const bool isq = w < qrows;
          const int wl = isq ? w : w - qrows;
          const int head = wl / dh, pi = wl - head * dh, jp = pi >> 1;  // pairs (v0,v1) -> jp, (v2,v3) -> jp+1
          if (o.rope) {
            const float2 cs0 = o.rope[(size_t)pos * half + jp], cs1 = o.rope[(size_t)pos * half + jp + 1];
            const float a0 = v0 * cs0.x - v1 * cs0.y, b0 = v1 * cs0.x + v0 * cs0.y;
            const float a1 = v2 * cs1.x - v3 * cs1.y, b1 = v3 * cs1.x + v2 * cs1.y;
            v0 = a0; v1 = b0; v2 = a1; v3 = b1;
          }
          bf16_t* base = isq ? o.q + (((size_t)b * o.H + head) * o.S + s) * dh
                             : o.k + (((size_t)b * o.Hkv + head) * o.S + s) * dh;
          *reinterpret_cast<uint32_t*>(base + jp) = (uint32_t)f2bf(v0) | ((uint32_t)f2bf(v2) << 16);
          *reinterpret_cast<uint32_t*>(base + half + jp) = (uint32_t)f2bf(v1) | ((uint32_t)f2bf(v3) << 16);
        } else {
          const int wl = w - qrows - krows;
          const int head = wl / dh, dd = wl - head * dh;
          bf16_t* base = o.vt + (((size_t)b * o.Hkv + head) * dh + dd) * o.Sp + s;
          base[0] = f2bf(v0);
          base[o.Sp] = f2bf(v1);
          base[2 * (size_t)o.Sp] = f2bf(v2);
          base[3 * (size_t)o.Sp] = f2bf(v3);
        }
      }
    }
  }
};

struct EpiF32 {
  float* out;
  template <int SW, int ST>
  __device__ void apply(f32x4_t (&acc)[SW][ST], int wb, int tb, int lane, int Nw, int T, int) const {
    const int wq = wb + 4 * (lane >> 4), tl = tb + (lane & 15);
#pragma unroll
    for (int j = 0; j < ST; ++j) {
      const int t = tl + 16 * j;
      if (t >= T) continue;
#pragma unroll
      for (int i = 0; i < SW; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int w = wq + 16 * i + r;
          if (w < Nw) out[(size_t)t * Nw + w] = acc[i][j][r];
        }
    }
  }
};

__device__ __forceinline__ bool better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}
struct Part {
  float m1, m2, s;
  int i1, i2;
};
__device__ __forceinline__ void top2_push(Part& p, float v, int id) {
  if (better(v, id, p.m1, p.i1)) {
    p.m2 = p.m1; p.i2 = p.i1; p.m1 = v; p.i1 = id;
  } else if (better(v, id, p.m2, p.i2)) {
    p.m2 = v; p.i2 = id;
  }
}
__device__ __forceinline__ Part part_merge(const Part& a, const Part& b) {
  Part o;
  if (better(a.m1, a.i1, b.m1, b.i1)) {
    o.m1 = a.m1; o.i1 = a.i1;
    if (better(a.m2, a.i2, b.m1, b.i1)) { o.m2 = a.m2; o.i2 = a.i2; } else { o.m2 = b.m1; o.i2 = b.i1; }
  } else {
    o.m1 = b.m1; o.i1 = b.i1;
    if (better(b.m2, b.i2, a.m1, a.i1)) { o.m2 = b.m2; o.i2 = b.i2; } else { o.m2 = a.m1; o.i2 = a.i1; }
  }
  // sums are relative to each side's own top-1 value
  const float sa = (a.m1 == -INFINITY) ? 0.f : a.s * __expf(a.m1 - o.m1);
  const float sb = (b.m1 == -INFINITY) ? 0.f : b.s * __expf(b.m1 - o.m1);
  o.s = sa + sb;
  return o;
}

// LM head: one partial per (token, vocabulary tile of BW ids). Within a wave: per-lane scan of its
// values, butterfly over the four lanes holding the same token, then a second pass for the sum of
// exp(l - m1_wave). Waves that split the tile's vocabulary rows merge through LDS in wave order.
template <int BW, int WW>
struct EpiLm {
  LmOut o;
  template <int SW, int ST>
  __device__ void apply(f32x4_t (&acc)[SW][ST], int wb, int tb, int lane, int Nw, int T, int tile_w) const {
    __shared__ Part xch[WW][256];  // [wave along W][token within the workgroup tile]; BT <= 256
    const int wid = threadIdx.x >> 6;
    const int wave_w = wid % WW, wave_t = wid / WW;
    const int R = *o.count;
    const int wq = wb + 4 * (lane >> 4), tl = tb + (lane & 15);
#pragma unroll
    for (int j = 0; j < ST; ++j) {
      Part p = {-INFINITY, -INFINITY, 0.f, INT_MAX, INT_MAX};
#pragma unroll
      for (int i = 0; i < SW; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int w = wq + 16 * i + r;
          if (w < Nw) top2_push(p, acc[i][j][r], w);
        }
#pragma unroll
      for (int off = 16; off <= 32; off <<= 1) {
        Part x;
        x.m1 = __shfl_xor(p.m1, off, 64); x.m2 = __shfl_xor(p.m2, off, 64);
        x.i1 = __shfl_xor(p.i1, off, 64); x.i2 = __shfl_xor(p.i2, off, 64);
        x.s = 0.f;
        Part y = (lane & off) ? part_merge(x, p) : part_merge(p, x);
        p.m1 = y.m1; p.m2 = y.m2; p.i1 = y.i1; p.i2 = y.i2;
      }
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < SW; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int w = wq + 16 * i + r;
          if (w < Nw) s += __expf(acc[i][j][r] - p.m1);
        }
      s += __shfl_xor(s, 16, 64);
      s += __shfl_xor(s, 32, 64);
      p.s = s;
      if (WW == 1) {
        const int t = tl + 16 * j;
        if (lane < 16 && t < R && t < T) {
          const size_t idx = (size_t)t * o.n_vt + tile_w;
          o.pm1[idx] = p.m1; o.pi1[idx] = p.i1; o.pm2[idx] = p.m2; o.pi2[idx] = p.i2; o.ps[idx] = p.s;
        }
      } else if (lane < 16) {
        xch[wave_w][(wave_t * ST + j) * 16 + lane] = p;
      }
    }
    if (WW > 1) {
      __syncthreads();
      if (wave_w == 0) {
#pragma unroll
        for (int j = 0; j < ST; ++j) {
          const int t = tl + 16 * j;
          if (lane < 16 && t < R && t < T) {
            Part p = xch[0][(wave_t * ST + j) * 16 + lane];
#pragma unroll
            for (int v = 1; v < WW; ++v) p = part_merge(p, xch[v][(wave_t * ST + j) * 16 + lane]);
            const size_t idx = (size_t)t * o.n_vt + tile_w;
            o.pm1[idx] = p.m1; o.pi1[idx] = p.i1; o.pm2[idx] = p.m2; o.pi2[idx] = p.i2; o.ps[idx] = p.s;
          }
        }
      }
    }
  }
};

// ---------------------------------------------------------------- the kernel
template <int BW, int BT, int WW, int WT, class Epi>
__global__ void __launch_bounds__(WW * WT * 64)
gemm_kernel(const bf16_t* __restrict__ W, const bf16_t* __restrict__ X, int Nw, int T, int K,
            const int32_t* __restrict__ t_count, Epi epi) {
  constexpr int NT = WW * WT * 64, TW = BW / WW, TT = BT / WT, SW = TW / 16, ST = TT / 16;
  constexpr int WCH = BW * 8, XCH = BT * 8;  // 16-byte chunks per stage
  constexpr int WPT = (WCH + NT - 1) / NT, XPT = (XCH + NT - 1) / NT;
  static_assert(TW % 16 == 0 && TT % 16 == 0, "wave tile must be a multiple of 16");
  extern __shared__ __attribute__((aligned(16))) bf16_t smem[];
  bf16_t* sW = smem;                      // [2][BW * LDSP]
  bf16_t* sX = smem + 2 * BW * LDSP;      // [2][BT * LDSP]

  // XCD-aware tile order: XCD x (= blockIdx % 8) walks a contiguous run of logical tiles; tiles
  // adjacent in that run share the weight tile and differ in the token tile.
  const int nW = (Nw + BW - 1) / BW, nTt = (T + BT - 1) / BT;
  const int total = nW * nTt;
  const int per = (total + 7) / 8;
  const int L = (blockIdx.x & 7) * per + (blockIdx.x >> 3);
  if (L >= total) return;
  const int tile_w = L / nTt, tile_t = L - tile_w * nTt;
  const int w0 = tile_w * BW, t0 = tile_t * BT;
  const int Tv = t_count ? min(T, *t_count) : T;  // valid token rows
  if (t0 >= Tv) return;

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wave_w = wid % WW, wave_t = wid / WW;

  f32x4_t acc[SW][ST];
#pragma unroll
  for (int i = 0; i < SW; ++i)
#pragma unroll
    for (int j = 0; j < ST; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  uint4 rw[WPT], rx[XPT];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < WPT; ++i) {
      const int c = tid + i * NT;
      const int row = c >> 3, col = (c & 7) * 8;
      const int gr = w0 + row, gk = k0 + col;
      rw[i] = (c < WCH && gr < Nw && gk < K) ? *reinterpret_cast<const uint4*>(W + (size_t)gr * K + gk)
                                             : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < XPT; ++i) {
      const int c = tid + i * NT;
      const int row = c >> 3, col = (c & 7) * 8;
      const int gt = t0 + row, gk = k0 + col;
      rx[i] = (c < XCH && gt < Tv && gk < K) ? *reinterpret_cast<const uint4*>(X + (size_t)gt * K + gk)
                                             : make_uint4(0, 0, 0, 0);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < WPT; ++i) {
      const int c = tid + i * NT;
      if (c < WCH) *reinterpret_cast<uint4*>(sW + buf * BW * LDSP + (c >> 3) * LDSP + (c & 7) * 8) = rw[i];
    }
#pragma unroll
    for (int i = 0; i < XPT; ++i) {
      const int c = tid + i * NT;
      if (c < XCH) *reinterpret_cast<uint4*>(sX + buf * BT * LDSP + (c >> 3) * LDSP + (c & 7) * 8) = rx[i];
    }
  };

  const int nk = (K + BK - 1) / BK;
  gload(0);
  sstore(0);
  __syncthreads();
  const int frag_row = lane & 15, frag_k = 8 * (lane >> 4);
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * BK);
    const bf16_t* cW = sW + cur * BW * LDSP + (wave_w * TW + frag_row) * LDSP + frag_k;
    const bf16_t* cX = sX + cur * BT * LDSP + (wave_t * TT + frag_row) * LDSP + frag_k;
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      bf16x8_t a[SW], b[ST];
#pragma unroll
      for (int i = 0; i < SW; ++i) a[i] = *reinterpret_cast<const bf16x8_t*>(cW + 16 * i * LDSP + 32 * ks);
#pragma unroll
      for (int j = 0; j < ST; ++j) b[j] = *reinterpret_cast<const bf16x8_t*>(cX + 16 * j * LDSP + 32 * ks);
#pragma unroll
      for (int i = 0; i < SW; ++i)
#pragma unroll
        for (int j = 0; j < ST; ++j) acc[i][j] = mfma16(a[i], b[j], acc[i][j]);
    }
    if (kt + 1 < nk) sstore(cur ^ 1);
    __syncthreads();
  }
  epi.template apply<SW, ST>(acc, w0 + wave_w * TW, t0 + wave_t * TT, lane, Nw, Tv, tile_w);
}

// ---------------------------------------------------------------- dispatch
template <int BW, int BT, int WW, int WT, class Epi>
static void run_gemm(const bf16_t* W, const bf16_t* X, int Nw, int T, int K, const int32_t* t_count, const Epi& epi,
                     hipStream_t s) {
  const int nW = (Nw + BW - 1) / BW, nTt = (T + BT - 1) / BT;
  const int total = nW * nTt;
  if (total == 0) return;
  const int grid = 8 * ((total + 7) / 8);
  const size_t lds = (size_t)2 * (BW + BT) * LDSP * sizeof(bf16_t);
  auto kern = gemm_kernel<BW, BT, WW, WT, Epi>;
  static bool attr_set = false;  // one kernel per instantiation; raise the dynamic-LDS cap once
  if (!attr_set) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    attr_set = true;
  }
  hipLaunchKernelGGL(kern, dim3(grid), dim3(WW * WT * 64), lds, s, W, X, Nw, T, K, t_count, epi);
}

// Tile choice: the large 128x128 tile when it yields enough workgroups to cover the 256 CUs,
// otherwise 128 weight rows x 64 tokens.
template <class Epi>
static void gemm_auto(const bf16_t* W, const bf16_t* X, int Nw, int T, int K, const Epi& epi, hipStream_t s) {
  const long big = (long)((Nw + 127) / 128) * ((T + 127) / 128);
  if (T > 64 && big >= 240)
    run_gemm<128, 128, 2, 2>(W, X, Nw, T, K, nullptr, epi, s);
  else
    run_gemm<128, 64, 2, 2>(W, X, Nw, T, K, nullptr, epi, s);
}

void gemm_qkv(const bf16_t* W, const bf16_t* X, int Nw, int T, int K, const QkvOut& o, hipStream_t s) {
  gemm_auto(W, X, Nw, T, K, EpiQkv{o}, s);
}
void gemm_resid(const bf16_t* W, const bf16_t* X, int Nw, int T, int K, float* r, hipStream_t s) {
  gemm_auto(W, X, Nw, T, K, EpiResid{r}, s);
}
void gemm_swiglu(const bf16_t* W, const bf16_t* X, int Nw, int T, int K, bf16_t* a, hipStream_t s) {
  gemm_auto(W, X, Nw, T, K, EpiSwiglu{a}, s);
}
void gemm_store_f32(const bf16_t* W, const bf16_t* X, int Nw, int T, int K, float* out, hipStream_t s) {
  gemm_auto(W, X, Nw, T, K, EpiF32{out}, s);
}
void gemm_lmhead(const bf16_t* W, const bf16_t* X, int V, int T, int K, const LmOut& o, hipStream_t s) {
  static_assert(kLmTile == 128, "LM-head tile is the GEMM's BW");
  if (T > 64)
    run_gemm<128, 128, 2, 2>(W, X, V, T, K, o.count, EpiLm<128, 2>{o}, s);
  else
    run_gemm<128, 64, 2, 2>(W, X, V, T, K, o.count, EpiLm<128, 2>{o}, s);
}

}  // namespace dcl
