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
//   LMHEAD per (token, 128-id vocabulary tile): top-1, top-2, sum exp(l - top1) and the entropy
//          sum — logits stay in registers and never reach memory;
//   PARTIAL float32 split-K slice, folded into the residual stream by the next RMSNorm;
//   F32    plain float32 store (debug logits).
// Tiles: BW weight rows x BT tokens per workgroup, K staged through a multi-stage LDS ring of
// 64- or 128-deep slices filled by direct-to-LDS DMA (gemm_kernel), or through registers
// (gemm_rp_kernel). The unit -> workgroup map is XCD-aware: consecutive tiles (which share a
// weight tile) land on the same XCD and its L2. The configuration of each GEMM shape comes from a
// measured table (gemm_tuned.inc), other shapes from a cost model.
#include <float.h>
#include <limits.h>

#include "dcl_internal.h"

namespace dcl {


__device__ __forceinline__ f32x4_t mfma16(const bf16x8_t& a, const bf16x8_t& b, const f32x4_t& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// ---------------------------------------------------------------- epilogues
// apply(): acc[i][j] holds C[wb + 16 i + 4 (lane/16) + r][tb + 16 j + lane%16], r = 0..3.

struct EpiResid {
  float* r;
  static constexpr bool kPartial = false;
  template <int SW, int ST>
  __device__ __forceinline__ void apply(f32x4_t (&acc)[SW][ST], int wb, int tb, int lane, int Nw, int T, int, int) const {
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
  static constexpr bool kPartial = false;
  template <int SW, int ST>
  __device__ __forceinline__ void apply(f32x4_t (&acc)[SW][ST], int wb, int tb, int lane, int Nw, int T, int, int) const {
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
        *reinterpret_cast<uint32_t*>(a + (size_t)t * F + (w >> 1)) = f2bf2(h0, h1);
      }
    }
  }
};

// Offsets are 32-bit element counts: gemm_qkv rejects outputs of 2^31 elements or more.
template <int DH>
struct EpiQkv {
  QkvOut o;
  static constexpr bool kPartial = false;
  template <int SW, int ST>
  __device__ __forceinline__ void apply(f32x4_t (&acc)[SW][ST], int wb, int tb, int lane, int Nw, int T, int, int) const {
    constexpr int HALF = DH / 2, LOG2DH = DH == 128 ? 7 : 6;
    static_assert(DH == 64 || DH == 128, "head_dim");
    const int qrows = o.H * DH, krows = o.Hkv * DH;
    const int Sk = o.Sk ? o.Sk : o.S;  // fresh key rows per (sequence, kv head); token s sits in slot koff + s
    const int wq = wb + 4 * (lane >> 4), tl = tb + (lane & 15);
#pragma unroll
    for (int j = 0; j < ST; ++j) {
      const int t = tl + 16 * j;
      if (t >= T) continue;
      const int b = t / o.S, s = t - b * o.S;
      const int pos = o.pos0 + s;
      // per token: element offsets of (head 0, position s) in q, k, and of (row 0, key s) in v^T
      const uint32_t qt = (uint32_t)(b * o.H * o.S + s) * DH;
      const uint32_t kt = (uint32_t)(b * o.Hkv * Sk + o.koff + s) * DH;
      const uint32_t vtt = (uint32_t)b * o.Hkv * DH * o.Sp + o.koff + s;
      const float2* rope_t = o.rope ? o.rope + (size_t)pos * HALF : nullptr;
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
          const int head = wl >> LOG2DH, jp = (wl & (DH - 1)) >> 1;  // pairs (v0,v1) -> jp, (v2,v3) -> jp+1
          if (rope_t) {
            const float2 cs0 = rope_t[jp], cs1 = rope_t[jp + 1];
            const float a0 = v0 * cs0.x - v1 * cs0.y, b0 = v1 * cs0.x + v0 * cs0.y;
            const float a1 = v2 * cs1.x - v3 * cs1.y, b1 = v3 * cs1.x + v2 * cs1.y;
            v0 = a0; v1 = b0; v2 = a1; v3 = b1;
          }
          bf16_t* base = isq ? o.q + qt + (uint32_t)head * o.S * DH : o.k + kt + (uint32_t)head * Sk * DH;
          *reinterpret_cast<uint32_t*>(base + jp) = f2bf2(v0, v2);
          *reinterpret_cast<uint32_t*>(base + HALF + jp) = f2bf2(v1, v3);
        } else {
          const int wl = w - qrows - krows;  // = head * DH + dimension
          bf16_t* base = o.vt + vtt + (uint32_t)wl * o.Sp;
          base[0] = f2bf(v0);
          base[o.Sp] = f2bf(v1);
          base[2 * o.Sp] = f2bf(v2);
          base[3 * o.Sp] = f2bf(v3);
          if (s == o.S - 1) {  // the last token also clears the padding slots [koff + S, Sp) of its four rows
            for (int z = 1; o.koff + s + z < o.Sp; ++z)
              for (int rr = 0; rr < 4; ++rr) base[rr * o.Sp + z] = 0;
          }
        }
      }
    }
  }
};

struct EpiF32 {
  float* out;
  static constexpr bool kPartial = false;
  template <int SW, int ST>
  __device__ __forceinline__ void apply(f32x4_t (&acc)[SW][ST], int wb, int tb, int lane, int Nw, int T, int, int) const {
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

// Split-K slice: unit `split` writes its float32 partial C to P + split * stride ([T, Nw] each);
// the consumer (the next RMSNorm) adds the slices to the residual stream in split order.
struct EpiPartial {
  float* P;
  size_t stride;
  static constexpr bool kPartial = true;
  template <int SW, int ST>
  __device__ __forceinline__ void apply(f32x4_t (&acc)[SW][ST], int wb, int tb, int lane, int Nw, int T, int,
                                        int split) const {
    float* base = P + (size_t)split * stride;
    const int wq = wb + 4 * (lane >> 4), tl = tb + (lane & 15);
#pragma unroll
    for (int j = 0; j < ST; ++j) {
      const int t = tl + 16 * j;
      if (t >= T) continue;
#pragma unroll
      for (int i = 0; i < SW; ++i) {
        const int w = wq + 16 * i;
        if (w >= Nw) continue;
        *reinterpret_cast<float4*>(base + (size_t)t * Nw + w) =
            make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
      }
    }
  }
};

__device__ __forceinline__ bool better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}
struct Part {
  float m1, m2, s, t;  // s = sum exp(l - m1), t = sum exp(l - m1) (l - m1), both relative to m1
  int i1, i2;
};
constexpr size_t kLmEpiLds = sizeof(Part) * kLmWaves * 256;  // static LDS of the LM-head epilogue
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
  // sums are relative to each side's own top-1 value; moving t to the new reference m adds
  // s (m1 - m) (each term exp(l - m1) (l - m1) becomes exp(l - m1) (l - m))
  const float da = (a.m1 == -INFINITY) ? 0.f : a.m1 - o.m1, db = (b.m1 == -INFINITY) ? 0.f : b.m1 - o.m1;
  const float ea = (a.m1 == -INFINITY) ? 0.f : __expf(da), eb = (b.m1 == -INFINITY) ? 0.f : __expf(db);
  o.s = a.s * ea + b.s * eb;
  o.t = ea * (a.t + a.s * da) + eb * (b.t + b.s * db);
  return o;
}

// LM head: one partial per (token, vocabulary tile of kLmTile ids). Within a wave: per-lane scan of
// its values, butterfly over the four lanes holding the same token, then a second pass for the sum
// of exp(l - m1_wave). A wave whose weight rows span a whole vocabulary tile (16 * SW == kLmTile)
// writes that tile's partial itself; otherwise the WW waves of a BW = kLmTile workgroup tile split
// its vocabulary rows and merge through LDS in wave order.
template <int BW, int WW>
struct EpiLm {
  LmOut o;
  static constexpr bool kPartial = false;
  // [wave along W][token within the workgroup tile] (BT <= 256); only the split-tile layout uses it
  __device__ static Part (*xch_slot())[256] {
    __shared__ Part xch[WW][256];
    return xch;
  }
  template <int SW, int ST>
  __device__ __forceinline__ void apply(f32x4_t (&acc)[SW][ST], int wb, int tb, int lane, int Nw, int T, int tile_w, int) const {
    constexpr bool kOwn = 16 * SW == kLmTile;  // this wave covers a whole vocabulary tile
    // any other layout is never planned for the LM head (plan_gemm's lm_ok); nothing to instantiate
    if constexpr (!kOwn && !(BW == kLmTile && 16 * SW * WW == BW)) return;
    const int wid = threadIdx.x >> 6;
    const int wave_w = wid % WW, wave_t = wid / WW;
    const int R = *o.count;
    const int vt = kOwn ? wb / kLmTile : tile_w;  // vocabulary tile of this wave's partial
    const int wq = wb + 4 * (lane >> 4), tl = tb + (lane & 15);
#pragma unroll
    for (int j = 0; j < ST; ++j) {
      Part p = {-INFINITY, -INFINITY, 0.f, 0.f, INT_MAX, INT_MAX};
#pragma unroll
      for (int i = 0; i < SW; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int w = wq + 16 * i + r;
          if (w < Nw && w != o.exclude) top2_push(p, acc[i][j][r], w);
        }
#pragma unroll
      for (int off = 16; off <= 32; off <<= 1) {
        Part x;
        x.m1 = __shfl_xor(p.m1, off, 64); x.m2 = __shfl_xor(p.m2, off, 64);
        x.i1 = __shfl_xor(p.i1, off, 64); x.i2 = __shfl_xor(p.i2, off, 64);
        x.s = 0.f;
        x.t = 0.f;
        Part y = part_merge(p, x);  // symmetric: ids differ, so argument order does not matter
        p.m1 = y.m1; p.m2 = y.m2; p.i1 = y.i1; p.i2 = y.i2;
      }
      float s = 0.f, t = 0.f;
#pragma unroll
      for (int i = 0; i < SW; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int w = wq + 16 * i + r;
          if (w < Nw && w != o.exclude) {
            const float d = acc[i][j][r] - p.m1;
            const float e = __expf(d);
            s += e;
            t += e * d;
          }
        }
      s += __shfl_xor(s, 16, 64);
      s += __shfl_xor(s, 32, 64);
      t += __shfl_xor(t, 16, 64);
      t += __shfl_xor(t, 32, 64);
      p.s = s;
      p.t = t;
      if constexpr (kOwn || WW == 1) {
        const int t = tl + 16 * j;
        if (lane < 16 && t < R && t < T && vt < o.n_vt) {
          const size_t idx = (size_t)t * o.n_vt + vt;
          o.pm1[idx] = p.m1; o.pi1[idx] = p.i1; o.pm2[idx] = p.m2; o.pi2[idx] = p.i2; o.ps[idx] = p.s;
          o.pt[idx] = p.t;
        }
      } else {
        if (lane < 16) xch_slot()[wave_w][(wave_t * ST + j) * 16 + lane] = p;
      }
    }
    if constexpr (!kOwn && WW > 1) {
      Part(*xch)[256] = xch_slot();
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
            o.pt[idx] = p.t;
          }
        }
      }
    }
  }
};

// ---------------------------------------------------------------- the kernel
// Direct-to-LDS multi-stage pipeline: each stage holds a BW x KD weight slice and a BT x KD
// activation slice (KD = 64 or 128 K elements), written by global_load_lds_dwordx4 (16 bytes per
// lane straight into LDS, no register staging). A row is KD/8 chunks of 16 bytes, XOR-swizzled
// (chunk c of row r at c ^ (r mod KD/8)) so the MFMA fragment reads are bank-conflict free.
// All STAGES buffers are in flight at once: buffer k mod STAGES is refilled with stage
// k + STAGES as soon as every wave holds stage k's fragments in registers. Fragments are double
// buffered per 32-wide K substep: the LDS reads of substep s + 1 are in flight while the MFMAs of
// substep s run, and the first substep of stage k + 1 is read across the stage boundary.
//
// The DMA instructions are issued through dma16_lds (inline assembly), so the compiler's wait-count
// pass does not treat them as pending LDS traffic and keeps its LDS waits fine-grained; their
// completion is tracked here with vmcnt waits on this wave's own
// outstanding stages, and a bare s_barrier (no vmcnt(0) fence) publishes a stage to the other
// waves. Vector-memory loads complete in issue order, and no other vector-memory load is issued
// inside the K loop, so "at most n outstanding" means "all but the newest n landed".
//
// Split-K: unit (tile, split) accumulates K-steps [split*per, ...) and hands its partial to a
// slice epilogue (EpiPartial: one float32 slice per split, no unit waits on another); the consumer
// adds the slices in split order, so results are bitwise reproducible. nsplit > 1 is only used with
// a slice epilogue.
__device__ __attribute__((aligned(64))) uint4 g_zero_chunk[4];

// dma16_at with the LDS destination already wave-uniform (a scalar register)
__device__ __forceinline__ void dma16_lds(const void* g, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds_addr), "v"(g) : "memory", "m0");
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

template <int BW, int BT, int KD, int STAGES, int WW, int WT, class Epi, bool KTAIL>
__global__ void __launch_bounds__(WW * WT * 64)
gemm_kernel(const bf16_t* __restrict__ W, const bf16_t* __restrict__ X, int Nw, int T, int K,
            const int32_t* __restrict__ t_count, int nsplit, Epi epi) {
  constexpr int NWAVE = WW * WT;
  constexpr int CPR = KD / 8, KS = KD / 32;  // 16-byte chunks per row, 32-wide substeps per stage
  constexpr int TW = BW / WW, TT = BT / WT, SW = TW / 16, ST = TT / 16;
  constexpr int CH = (BW + BT) * CPR;        // chunks per stage
  constexpr int IPW = CH / 64 / NWAVE;       // load instructions per wave per stage
  static_assert(TW % 16 == 0 && TT % 16 == 0 && CH % (64 * NWAVE) == 0 && (BW * CPR) % 64 == 0, "tile shape");
  static_assert((KD == 64 || KD == 128) && STAGES >= 2 && IPW * (STAGES - 1) < 64, "pipeline shape");
  extern __shared__ __attribute__((aligned(1024))) uint4 sm[];

  // Units: (split, weight tile, token tile), token tile innermost so neighbours share a weight
  // slice, split outermost so an XCD's run covers one or two K ranges and its L2 holds only that
  // part of the activations. Only token tiles holding valid rows (t_count, when given) are units.
  // XCD x (= blockIdx % 8) walks a contiguous run of units, its workgroups striding through it.
  const int Tv = t_count ? min(T, *t_count) : T;
  const int nW = (Nw + BW - 1) / BW, nTt = (Tv + BT - 1) / BT;
  const int units = nW * nsplit * nTt;
  const int per = (units + 7) / 8;
  const int xcd = blockIdx.x & 7, stride = gridDim.x >> 3;
  const int run_end = min(units, (xcd + 1) * per);
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wave_w = wid % WW, wave_t = wid / WW;
  const int frow = lane & 15, fchunk = lane >> 4;
  for (int L = xcd * per + (blockIdx.x >> 3); L < run_end; L += stride) {
    const int tile_t = L % nTt, rest = L / nTt;
    const int tile_w = rest % nW, split = rest / nW;
    const int w0 = tile_w * BW, t0 = tile_t * BT;
    const int nk_all = (K + KD - 1) / KD;
    const int kper = (nk_all + nsplit - 1) / nsplit;
    const int kb = min(nk_all, split * kper);
    const int nk = min(nk_all, kb + kper) - kb;

    // Per-lane source of this wave's load instructions at K offset 0. A row outside the operand
    // is clamped to the last valid row: its data only reaches accumulators of rows / tokens that
    // every epilogue skips, so no zero fill is needed. The source of stage kt is this pointer plus
    // (kb + kt) * KD elements; with KTAIL (K not a multiple of KD), chunks past K read the zero chunk.
    const bf16_t* gsrc[IPW];
    int kc[IPW];
#pragma unroll
    for (int i = 0; i < IPW; ++i) {
      const int q = wid * IPW + i;
      const int pos = q * 64 + lane;
      const bool isw = q * 64 < BW * CPR;
      const int p2 = isw ? pos : pos - BW * CPR;
      const int row = p2 / CPR, c = (p2 % CPR) ^ (row & (CPR - 1));
      const int grow = min((isw ? w0 : t0) + row, (isw ? Nw : Tv) - 1);
      gsrc[i] = (isw ? W : X) + (size_t)grow * K + c * 8;
      kc[i] = c * 8;
    }
    const uint32_t lds0 = lds_addr_of(sm) + (uint32_t)(__builtin_amdgcn_readfirstlane(wid) * IPW) * 1024u;
    auto issue = [&](int kt) {
      const uint32_t stage = lds0 + (uint32_t)((kt % STAGES) * CH) * 16u;
      const int k0 = (kb + kt) * KD;
#pragma unroll
      for (int i = 0; i < IPW; ++i) {
        const bf16_t* g = gsrc[i] + k0;
        if constexpr (KTAIL)
          if (k0 + kc[i] >= K) g = reinterpret_cast<const bf16_t*>(g_zero_chunk);
        dma16_lds(g, stage + (uint32_t)i * 1024u);
      }
    };
    auto frag = [&](int kt, int ks, bf16x8_t(&a)[SW], bf16x8_t(&b)[ST]) {
      const uint4* stage = sm + (kt % STAGES) * CH;
      const int c = 4 * ks + fchunk;
#pragma unroll
      for (int i = 0; i < SW; ++i) {
        const int r = wave_w * TW + 16 * i + frow;
        a[i] = __builtin_bit_cast(bf16x8_t, stage[r * CPR + (c ^ (r & (CPR - 1)))]);
      }
#pragma unroll
      for (int j = 0; j < ST; ++j) {
        const int r = wave_t * TT + 16 * j + frow;
        b[j] = __builtin_bit_cast(bf16x8_t, stage[BW * CPR + r * CPR + (c ^ (r & (CPR - 1)))]);
      }
    };
    f32x4_t acc[SW][ST];
#pragma unroll
    for (int i = 0; i < SW; ++i)
#pragma unroll
      for (int j = 0; j < ST; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    auto mma = [&](const bf16x8_t(&a)[SW], const bf16x8_t(&b)[ST]) {
#pragma unroll
      for (int i = 0; i < SW; ++i)
#pragma unroll
        for (int j = 0; j < ST; ++j) acc[i][j] = mfma16(a[i], b[j], acc[i][j]);
    };

    auto mma_rows = [&](const bf16x8_t(&a)[SW], const bf16x8_t(&b)[ST], int i0, int i1) {
#pragma unroll
      for (int i = 0; i < SW; ++i)
        if (i >= i0 && i < i1)
#pragma unroll
          for (int j = 0; j < ST; ++j) acc[i][j] = mfma16(a[i], b[j], acc[i][j]);
    };
#pragma unroll
    for (int st = 0; st < STAGES; ++st)
      if (st < nk) issue(st);
    {  // stage 0 landed; stages 1 .. min(nk, STAGES) - 1 may still fly
      const int pend = min(STAGES - 1, nk - 1);
      if (STAGES >= 3 && pend >= 2) wait_vmcnt<(STAGES >= 3 ? 2 : 0) * IPW>();
      else if (pend >= 1) wait_vmcnt<IPW>();
      else wait_vmcnt<0>();
    }
    lds_barrier();
    bf16x8_t fa[2][SW], fb[2][ST];
    if (nk > 0) frag(0, 0, fa[0], fb[0]);
    for (int kt = 0; kt + 1 < nk; ++kt) {
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        if (s + 1 < KS) {
          frag(kt, s + 1, fa[(s + 1) & 1], fb[(s + 1) & 1]);
        } else {
          // stage kt + 1 landed (stages kt + 2 .. min(nk - 1, kt + STAGES - 1) may still fly);
          // after the barrier every wave holds stage kt in registers, so its buffer is refilled
          const int pend = min(STAGES - 2, nk - 2 - kt);
          if (STAGES >= 4 && pend >= 2) wait_vmcnt<(STAGES >= 4 ? 2 : 0) * IPW>();
          else if (STAGES >= 3 && pend >= 1) wait_vmcnt<(STAGES >= 3 ? 1 : 0) * IPW>();
          else wait_vmcnt<0>();
          lds_barrier();
          if constexpr (STAGES >= 3) {
            // the next stage's first fragments go out first, and the refill is issued between two
            // halves of this substep's MFMAs, so its address work overlaps the matrix pipe
            frag(kt + 1, 0, fa[0], fb[0]);
            mma_rows(fa[s & 1], fb[s & 1], 0, (SW + 1) / 2);
            if (kt + STAGES < nk) issue(kt + STAGES);
            mma_rows(fa[s & 1], fb[s & 1], (SW + 1) / 2, SW);
            continue;
          } else {
            // one stage in flight: the refill goes out at once, ahead of everything else
            if (kt + STAGES < nk) issue(kt + STAGES);
            frag(kt + 1, 0, fa[0], fb[0]);
          }
        }
        mma(fa[s & 1], fb[s & 1]);
      }
    }
    if (nk > 0) {
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        if (s + 1 < KS) frag(nk - 1, s + 1, fa[(s + 1) & 1], fb[(s + 1) & 1]);
        mma(fa[s & 1], fb[s & 1]);
      }
    }

    epi.template apply<SW, ST>(acc, w0 + wave_w * TW, t0 + wave_t * TT, lane, Nw, Tv, tile_w, split);
    lds_barrier();  // the next unit's prologue overwrites LDS the epilogue may still read
  }
}

// Register-prefetch variant: global -> VGPR loads run PF stages ahead of the MFMAs (the data in
// flight sits in registers, not in LDS), each stage is written into a double-buffered,
// XOR-swizzled LDS tile just before it is needed. The compiler's vmcnt waits cover exactly the
// stage being stored. Same unit order, split-K slices and epilogues as gemm_kernel.
template <int BW, int BT, int PF, int WW, int WT, class Epi>
__global__ void __launch_bounds__(WW * WT * 64)
gemm_rp_kernel(const bf16_t* __restrict__ W, const bf16_t* __restrict__ X, int Nw, int T, int K,
               const int32_t* __restrict__ t_count, int nsplit, Epi epi) {
  constexpr int NWAVE = WW * WT, NT = NWAVE * 64;
  constexpr int TW = BW / WW, TT = BT / WT, SW = TW / 16, ST = TT / 16;
  constexpr int CH = (BW + BT) * 8;   // 16-byte chunks per stage
  constexpr int CPT = CH / NT;        // chunks per thread per stage
  static_assert(TW % 16 == 0 && TT % 16 == 0 && CH % NT == 0, "tile shape");
  extern __shared__ __attribute__((aligned(1024))) uint4 sm[];

  const int nW = (Nw + BW - 1) / BW, nTt = (T + BT - 1) / BT;
  const int tiles = nW * nTt, units = tiles * nsplit;
  const int per = (units + 7) / 8;
  const int L = (blockIdx.x & 7) * per + (blockIdx.x >> 3);
  if (L >= units) return;
  const int tile_t = L % nTt, rest = L / nTt;
  const int tile_w = rest % nW, split = rest / nW;
  const int tile = tile_w * nTt + tile_t;
  const int w0 = tile_w * BW, t0 = tile_t * BT;
  const int Tv = t_count ? min(T, *t_count) : T;
  if (t0 >= Tv) return;
  const int nk_all = (K + 63) / 64;
  const int kper = (nk_all + nsplit - 1) / nsplit;
  const int kb = min(nk_all, split * kper);
  const int nk = min(nk_all, kb + kper) - kb;

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wave_w = wid % WW, wave_t = wid / WW;

  // chunk j of this thread: stage position pos = j * NT + tid; source pointer (null = zero chunk)
  const bf16_t* src[CPT];
  int lds_pos[CPT];
  int kcol[CPT];
#pragma unroll
  for (int j = 0; j < CPT; ++j) {
    const int pos = j * NT + tid;
    const bool isw = pos < BW * 8;
    const int p2 = isw ? pos : pos - BW * 8;
    const int row = p2 >> 3, c = p2 & 7;
    const int grow = (isw ? w0 : t0) + row;
    src[j] = (grow < (isw ? Nw : Tv)) ? (isw ? W : X) + (size_t)grow * K + c * 8 : nullptr;
    kcol[j] = c * 8;
    lds_pos[j] = (isw ? 0 : BW * 8) + row * 8 + (c ^ (row & 7));
  }
  uint4 regs[PF][CPT];
  auto gload = [&](int set, int kt) {
    const int k0 = (kb + kt) * 64;
#pragma unroll
    for (int j = 0; j < CPT; ++j)
      regs[set][j] = (src[j] && k0 + kcol[j] < K) ? *reinterpret_cast<const uint4*>(src[j] + k0) : make_uint4(0, 0, 0, 0);
  };
  auto sstore = [&](int set, int buf) {
    uint4* stage = sm + buf * CH;
#pragma unroll
    for (int j = 0; j < CPT; ++j) stage[lds_pos[j]] = regs[set][j];
  };

  f32x4_t acc[SW][ST];
#pragma unroll
  for (int i = 0; i < SW; ++i)
#pragma unroll
    for (int j = 0; j < ST; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int st = 0; st < PF; ++st)
    if (st < nk) gload(st, st);
  if (nk > 0) sstore(0, 0);
  lds_barrier();
  const int frow = lane & 15, fchunk = lane >> 4;
  auto compute = [&](int buf) {
    const uint4* stage = sm + buf * CH;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int c = 4 * ks + fchunk;
      bf16x8_t a[SW], b[ST];
#pragma unroll
      for (int i = 0; i < SW; ++i) {
        const int r = wave_w * TW + 16 * i + frow;
        a[i] = __builtin_bit_cast(bf16x8_t, stage[r * 8 + (c ^ (r & 7))]);
      }
#pragma unroll
      for (int j = 0; j < ST; ++j) {
        const int r = wave_t * TT + 16 * j + frow;
        b[j] = __builtin_bit_cast(bf16x8_t, stage[BW * 8 + r * 8 + (c ^ (r & 7))]);
      }
#pragma unroll
      for (int i = 0; i < SW; ++i)
#pragma unroll
        for (int j = 0; j < ST; ++j) acc[i][j] = mfma16(a[i], b[j], acc[i][j]);
    }
  };
  // main loop, unrolled by PF so register-set indices are compile-time constants
  for (int kt0 = 0; kt0 < nk; kt0 += PF) {
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      const int kt = kt0 + u;
      if (kt < nk) {
        if (kt + PF < nk) gload(u, kt + PF);          // set u held stage kt, already in LDS
        compute(kt & 1);
        if (kt + 1 < nk) sstore((u + 1) % PF, (kt + 1) & 1);
        lds_barrier();
      }
    }
  }

  if constexpr (Epi::kPartial) {
    epi.template apply<SW, ST>(acc, w0 + wave_w * TW, t0 + wave_t * TT, lane, Nw, Tv, tile_w, split);
    return;
  }
  epi.template apply<SW, ST>(acc, w0 + wave_w * TW, t0 + wave_t * TT, lane, Nw, Tv, tile_w, split);
}

template <int BW, int BT, int PF, class Epi, int WW = 2, int WT = 2>
static void run_rp(const bf16_t* W, const bf16_t* X, int Nw, int T, int K, const int32_t* t_count, int nsplit,
                   const Epi& epi, hipStream_t s) {
  const int tiles = ((Nw + BW - 1) / BW) * ((T + BT - 1) / BT);
  const int units = tiles * nsplit;
  if (units == 0) return;
  const int grid = 8 * ((units + 7) / 8);
  const size_t lds = (size_t)2 * (BW + BT) * 8 * 16;
  auto kern = gemm_rp_kernel<BW, BT, PF, WW, WT, Epi>;
  static std::atomic<uint32_t> lds_set{0};
  ensure_dynamic_lds(reinterpret_cast<const void*>(kern), lds, lds_set);
  hipLaunchKernelGGL(kern, dim3(grid), dim3(WW * WT * 64), lds, s, W, X, Nw, T, K, t_count, nsplit, epi);
}

// ---------------------------------------------------------------- planning and dispatch
struct TileCfg {
  int bw, bt, kd, stages, ww, wt, rp;  // rp = 1: register-prefetch kernel, `stages` = prefetch depth
};
// Tile shapes (weight rows x tokens), K depth per stage, stages and wave grid, chosen among by
// measurement on MI355X for the LLaDA / Dream shapes (the tuned table below). A K depth of 128
// halves the number of stage handoffs, which is what limits the small-tile shapes; 8-16 waves per
// workgroup keep the MFMA pipes busy while the LDS fragment reads of the next substep are in
// flight.
static const TileCfg kCfgs[] = {
    {128, 128, 64, 2, 2, 4, 0},  {192, 192, 64, 3, 4, 2, 0},  {64, 64, 64, 4, 2, 2, 0},
    {128, 256, 64, 3, 2, 4, 0},  {96, 192, 64, 3, 2, 2, 1},   {192, 192, 64, 2, 4, 2, 1},
    {128, 128, 64, 3, 2, 4, 1},  {96, 192, 128, 2, 3, 4, 0},  {128, 96, 128, 2, 4, 2, 0},
    {160, 128, 128, 2, 2, 4, 0}, {96, 192, 128, 2, 2, 4, 0},  {192, 192, 64, 3, 4, 4, 0},
    {128, 128, 128, 2, 2, 4, 0}, {64, 192, 128, 2, 2, 4, 0},  {128, 192, 128, 2, 4, 4, 0},
    {128, 128, 64, 3, 2, 4, 0},  {128, 256, 64, 3, 2, 8, 0},  {128, 192, 64, 3, 2, 4, 0},
    {128, 256, 64, 2, 2, 8, 0},  {256, 256, 64, 2, 2, 4, 0},  {256, 192, 64, 2, 2, 4, 0},
    {256, 128, 64, 3, 2, 2, 0},  {256, 256, 64, 2, 4, 2, 0},  {96, 192, 64, 4, 3, 4, 0},
    {96, 192, 64, 3, 3, 4, 0},   {192, 96, 64, 3, 4, 3, 0},
};
constexpr int kNumCfgs = sizeof(kCfgs) / sizeof(kCfgs[0]);
constexpr int kCUs = 256;
constexpr size_t kLdsBytes = 160 * 1024;  // LDS per CU (gfx950)

// Measured choices for the GEMM shapes of the LLaDA-8B / Dream-7B workloads (weight rows, tokens, K).
struct TunedShape {
  int nw, t, k, cfg, nsplit;
};
static const TunedShape kTuned[] = {
#include "gemm_tuned.inc"
};

static size_t cfg_lds(const TileCfg& c) {
  return c.rp ? (size_t)2 * (c.bw + c.bt) * 8 * 16 : (size_t)c.stages * (c.bw + c.bt) * (c.kd / 8) * 16;
}

// Fallback estimate for shapes outside the table: saturated throughput of the configuration, or the
// time of one workgroup when there are fewer workgroups than CUs.
static double plan_cost(const TileCfg& c, int n, int Nw, int T, int K) {
  const double tiles = (double)((Nw + c.bw - 1) / c.bw) * ((T + c.bt - 1) / c.bt);
  const double units = tiles * n;
  const int bpc = (int)(160 * 1024 / cfg_lds(c)) > 0 ? (int)(160 * 1024 / cfg_lds(c)) : 1;
  const double sw = c.bw / 32.0, st = c.bt / 32.0;
  const double eff = sw * st / (sw * st + 0.5 * (sw + st));
  const double mac_rate = 2.5e15 / 2 / kCUs * 0.3;  // sustained MAC/s per CU
  const double t_unit = (double)c.bw * c.bt * ((double)K / n) / eff / mac_rate;
  const double slots = (double)kCUs * (bpc < 2 ? 1 : 2);
  const double t_part = n > 1 ? 2.0 * (n - 1) * (double)T * Nw * 4 / 6e12 : 0.0;
  return ceil(units / slots) * t_unit * (bpc < 2 ? 1.0 : 1.6) + t_part;
}

// force_bw != 0 (the LM head): the tile must be force_bw weight rows split over exactly
// kLmWaves waves along W, the layout the top-2 epilogue's cross-wave merge is written for.
static bool lm_ok(const TileCfg& c, int force_bw) {
  if (!force_bw || c.rp) return !force_bw;
  if (c.bw / c.ww == force_bw) return cfg_lds(c) <= kLdsBytes;  // each wave owns a vocabulary tile
  return c.bw == force_bw && c.ww == kLmWaves && cfg_lds(c) + kLmEpiLds <= kLdsBytes;
}

GemmPlan plan_gemm(int Nw, int T, int K, int force_bw, int max_split) {
  GemmPlan best{0, 1, 0};
  bool found = false;
  for (const TunedShape& ts : kTuned)
    if (ts.nw == Nw && ts.t == T && ts.k == K && ts.nsplit <= max_split && lm_ok(kCfgs[ts.cfg], force_bw)) {
      best.cfg = ts.cfg;
      best.nsplit = ts.nsplit;
      found = true;
      break;
    }
  if (!found) {
    double best_t = 1e30;
    const int nk = (K + 63) / 64;
    for (int ci = 0; ci < kNumCfgs; ++ci) {
      if (!lm_ok(kCfgs[ci], force_bw)) continue;
      for (int n = 1; n <= max_split; ++n) {
        if (n > 1 && nk / n < 8) break;
        const double t = plan_cost(kCfgs[ci], n, Nw, T, K);
        if (t < best_t * 0.999) {
          best_t = t;
          best.cfg = ci;
          best.nsplit = n;
        }
      }
    }
  }
  // K not a multiple of the plan's stage depth: one tail-aware configuration (128 x 128, 64-deep stages,
  // which also suits the LM head's split layout) serves every such shape, none of the tuned model
  // shapes, so the tuned kernels carry no tail handling; the register-prefetch kernel handles tails itself
  if (!kCfgs[best.cfg].rp && K % kCfgs[best.cfg].kd != 0) best.cfg = 0;
  const TileCfg& c = kCfgs[best.cfg];
  best.tiles = ((Nw + c.bw - 1) / c.bw) * ((T + c.bt - 1) / c.bt);
  return best;
}

void gemm_cfg_shape(int cfg, int* shape) {
  const TileCfg& c = kCfgs[cfg >= 0 && cfg < kNumCfgs ? cfg : 0];
  shape[0] = c.bw;
  shape[1] = c.bt;
  shape[2] = c.kd;
  shape[3] = c.stages;
  shape[4] = c.ww;
  shape[5] = c.wt;
}

template <int BW, int BT, int KD, int STAGES, int WW, int WT, class Epi, bool KTAIL = false>
static void run_cfg(const bf16_t* W, const bf16_t* X, int Nw, int T, int K, const int32_t* t_count, int nsplit,
                    const Epi& epi, hipStream_t s) {
  const int tiles = ((Nw + BW - 1) / BW) * ((T + BT - 1) / BT);
  const int units = tiles * nsplit;
  if (units == 0) return;
  // One workgroup per unit; with a device-side row count the grid is capped (workgroups stride
  // over the units that turn out to be active) so inactive token tiles cost no dispatch.
  int grid = 8 * ((units + 7) / 8);
  if (t_count && grid > 8 * kCUs) grid = 8 * kCUs;
  const size_t lds = (size_t)STAGES * (BW + BT) * (KD / 8) * 16;
  auto kern = gemm_kernel<BW, BT, KD, STAGES, WW, WT, Epi, KTAIL>;
  // per instantiation: the ring plus the epilogue's static LDS fit in a CU (-1 = not yet known)
  static std::atomic<int> fits{-1};
  if (fits.load(std::memory_order_acquire) < 0) {
    hipFuncAttributes at{};
    fits.store(hipFuncGetAttributes(&at, reinterpret_cast<const void*>(kern)) == hipSuccess &&
                   at.sharedSizeBytes + lds <= kLdsBytes,
               std::memory_order_release);
  }
  // A ring that does not fit is never planned (plans respect kLdsBytes). Rather than a launch the runtime
  // would reject, the smallest configuration runs; that one always fits and is launched even if the
  // attribute query itself failed, so this never recurses.
  constexpr bool kSmallest = BW == 128 && BT == 128 && KD == 64 && STAGES == 2 && WW == 2 && WT == 4;
  if constexpr (!kSmallest) {
    if (!fits.load(std::memory_order_acquire)) {
      run_cfg<128, 128, 64, 2, 2, 4, Epi, KTAIL>(W, X, Nw, T, K, t_count, nsplit, epi, s);
      return;
    }
  }
  static std::atomic<uint32_t> lds_set{0};
  ensure_dynamic_lds(reinterpret_cast<const void*>(kern), lds, lds_set);
  hipLaunchKernelGGL(kern, dim3(grid), dim3(WW * WT * 64), lds, s, W, X, Nw, T, K, t_count, nsplit, epi);
}

static_assert(kNumCfgs == 26, "run_plan dispatches every configuration of kCfgs");

template <class Epi>
static void run_plan(const GemmPlan& p, const bf16_t* W, const bf16_t* X, int Nw, int T, int K, const int32_t* t_count,
                     const Epi& epi, hipStream_t s) {
  const int n = p.nsplit;
  if (!kCfgs[p.cfg].rp && K % kCfgs[p.cfg].kd != 0) {  // plan_gemm gives such shapes configuration 0
    run_cfg<128, 128, 64, 2, 2, 4, Epi, true>(W, X, Nw, T, K, t_count, n, epi, s);
    return;
  }
  switch (p.cfg) {
    case 0: run_cfg<128, 128, 64, 2, 2, 4>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 1: run_cfg<192, 192, 64, 3, 4, 2>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 2: run_cfg<64, 64, 64, 4, 2, 2>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 3: run_cfg<128, 256, 64, 3, 2, 4>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 4: run_rp<96, 192, 3, Epi, 2, 2>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 5: run_rp<192, 192, 2, Epi, 4, 2>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 6: run_rp<128, 128, 3, Epi, 2, 4>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 7: run_cfg<96, 192, 128, 2, 3, 4>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 8: run_cfg<128, 96, 128, 2, 4, 2>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 9: run_cfg<160, 128, 128, 2, 2, 4>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 10: run_cfg<96, 192, 128, 2, 2, 4>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 11: run_cfg<192, 192, 64, 3, 4, 4>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 12: run_cfg<128, 128, 128, 2, 2, 4>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 13: run_cfg<64, 192, 128, 2, 2, 4>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 14: run_cfg<128, 192, 128, 2, 4, 4>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 15: run_cfg<128, 128, 64, 3, 2, 4>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 16: run_cfg<128, 256, 64, 3, 2, 8>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 17: run_cfg<128, 192, 64, 3, 2, 4>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 18: run_cfg<128, 256, 64, 2, 2, 8>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 19: run_cfg<256, 256, 64, 2, 2, 4>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 20: run_cfg<256, 192, 64, 2, 2, 4>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 21: run_cfg<256, 128, 64, 3, 2, 2>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 22: run_cfg<256, 256, 64, 2, 4, 2>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 23: run_cfg<96, 192, 64, 4, 3, 4>(W, X, Nw, T, K, t_count, n, epi, s); break;
    case 24: run_cfg<96, 192, 64, 3, 3, 4>(W, X, Nw, T, K, t_count, n, epi, s); break;
    default: run_cfg<192, 96, 64, 3, 4, 3>(W, X, Nw, T, K, t_count, n, epi, s); break;
  }
}

void gemm_qkv(const bf16_t* W, const bf16_t* X, int Nw, int T, int K, const QkvOut& o, hipStream_t s) {
  const GemmPlan p = plan_gemm(Nw, T, K, 0, 1);
  if (o.dh == 128) run_plan(p, W, X, Nw, T, K, nullptr, EpiQkv<128>{o}, s);
  else run_plan(p, W, X, Nw, T, K, nullptr, EpiQkv<64>{o}, s);
}
int gemm_resid(const bf16_t* W, const bf16_t* X, int Nw, int T, int K, float* r, float* P, hipStream_t s) {
  const GemmPlan p = plan_gemm(Nw, T, K, 0, P ? kMaxSplit : 1);
  if (p.nsplit > 1) {
    run_plan(p, W, X, Nw, T, K, nullptr, EpiPartial{P, (size_t)T * Nw}, s);
    return p.nsplit;
  }
  run_plan(p, W, X, Nw, T, K, nullptr, EpiResid{r}, s);
  return 0;
}
void gemm_swiglu(const bf16_t* W, const bf16_t* X, int Nw, int T, int K, bf16_t* a, hipStream_t s) {
  run_plan(plan_gemm(Nw, T, K, 0, 1), W, X, Nw, T, K, nullptr, EpiSwiglu{a}, s);
}
void gemm_store_f32(const bf16_t* W, const bf16_t* X, int Nw, int T, int K, float* out, hipStream_t s) {
  run_plan(plan_gemm(Nw, T, K, 0, 1), W, X, Nw, T, K, nullptr, EpiF32{out}, s);
}
void gemm_lmhead(const bf16_t* W, const bf16_t* X, int V, int T, int K, const LmOut& o, hipStream_t s) {
  static_assert(kLmTile == 128 && kLmWaves == 2, "the LM-head vocabulary tile is the GEMM's weight tile");
  run_plan(plan_gemm(V, T, K, kLmTile, 1), W, X, V, T, K, o.count, EpiLm<kLmTile, kLmWaves>{o}, s);
}

}  // namespace dcl
