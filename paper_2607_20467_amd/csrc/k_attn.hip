// Non-causal (bidirectional) flash-style attention for gfx950, MHA and GQA, head_dim 64 / 128.
//
// Masked diffusion LMs attend from every position to every position; there is no causal mask, so
// the whole S x S score matrix is real work. One workgroup handles 16*NW queries of one (batch,
// head); each wavefront owns 16 queries and walks the keys in tiles of 64 with an online softmax
// in float32. Keys are [cached prefix (P) || the S fresh tokens].
//
// Orientation: the score tile is computed transposed, S^T = K Q^T (MFMA A = K from LDS, B = Q held
// in registers), so each lane holds 16 scores of ONE query. Its softmax probabilities then feed the
// P*V product directly as the MFMA B operand of O^T = V^T P^T, with V^T read from a key-contiguous
// LDS tile in the matching key order; no register shuffle of P is needed.
// P is split into bf16 hi + lo parts (two MFMAs), so the probabilities enter the product with
// ~16 significant bits instead of 8.
#include "dcl_internal.h"

namespace dcl {

constexpr int KT = 64;  // keys per tile

__device__ __attribute__((aligned(64))) uint4 g_attn_zero[4];

__device__ __forceinline__ f32x4_t mfma16a(const bf16x8_t& a, const bf16x8_t& b, const f32x4_t& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// op(v, v of lane ^ 16) and op(v, v of lane ^ 32) in every lane, through the gfx950 lane-swap
// instructions (no LDS round trip). The swap of a register with itself leaves, per lane, the
// value of both partners in the two results; op must be commutative.
template <class Op>
__device__ __forceinline__ float xor_lanes16(float v, Op op) {
  const int b = __builtin_bit_cast(int, v);
  const auto p = __builtin_amdgcn_permlane16_swap(b, b, false, false);
  return op(__builtin_bit_cast(float, (int)p[0]), __builtin_bit_cast(float, (int)p[1]));
}
template <class Op>
__device__ __forceinline__ float xor_lanes32(float v, Op op) {
  const int b = __builtin_bit_cast(int, v);
  const auto p = __builtin_amdgcn_permlane32_swap(b, b, false, false);
  return op(__builtin_bit_cast(float, (int)p[0]), __builtin_bit_cast(float, (int)p[1]));
}

template <int N>
__device__ __forceinline__ void attn_wait_vmcnt() {
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// K and V^T tiles move HBM/L2 -> LDS with global_load_lds_dwordx4 into a STAGES-deep ring (no
// register staging, no padding). K rows (DH/8 chunks of 16 bytes) are XOR-swizzled by the key
// index, V^T rows (8 chunks = 64 keys) by the dimension index, so the fragment reads below are
// bank-conflict free. Chunks past the last key read a zero chunk.
template <int NW, int DH, int STAGES>
__global__ void __launch_bounds__(NW * 64) attn_kernel(AttnArgs a) {
  constexpr int BQ = 16 * NW, NT = NW * 64;
  constexpr int KC = DH / 8;           // chunks per K row
  constexpr int KCH = KT * KC;         // K chunks per stage
  constexpr int VCH = DH * (KT / 8);   // V^T chunks per stage
  constexpr int SCH = KCH + VCH;       // chunks per stage
  constexpr int IPW = SCH / 64 / NW;   // load instructions per wave per stage
  static_assert(SCH % (64 * NW) == 0 && KCH % 64 == 0, "stage shape");
  extern __shared__ __attribute__((aligned(1024))) uint4 sm[];

  // Units (batch, head, query tile), query tile innermost: XCD x (= blockIdx % 8) takes a contiguous
  // run of units, so the query tiles of one head (and the heads sharing a KV head) read their keys
  // and values through one L2.
  const int nqt = (a.S + BQ - 1) / BQ;
  const int units = nqt * a.H * a.B, per = (units + 7) / 8;
  const int L = (blockIdx.x & 7) * per + (blockIdx.x >> 3);
  if (L >= units) return;
  const int qt = L % nqt, h = (L / nqt) % a.H, b = L / (nqt * a.H);
  const int g = h / (a.H / a.Hkv);
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int lq = lane & 15, lg = lane >> 4;
  const int S = a.S, P = a.P, nkeys = P + S;
  const int qrow = qt * BQ + wid * 16 + lq;
  const int ntiles = (nkeys + KT - 1) / KT;

  bf16x8_t qf[DH / 32];
  {
    const bf16_t* qp = a.q + (((size_t)b * a.H + h) * S + (qrow < S ? qrow : 0)) * DH + 8 * lg;
#pragma unroll
    for (int ks = 0; ks < DH / 32; ++ks) {
      uint4 v = qrow < S ? *reinterpret_cast<const uint4*>(qp + 32 * ks) : make_uint4(0, 0, 0, 0);
      qf[ks] = __builtin_bit_cast(bf16x8_t, v);
    }
  }
  const size_t kvh = (size_t)b * a.Hkv + g;
  const bf16_t* kc = a.kc ? a.kc + kvh * a.Pc * DH : nullptr;
  const bf16_t* kf = a.k + kvh * S * DH;
  const bf16_t* vc = a.vc ? a.vc + kvh * DH * a.Pc : nullptr;
  const bf16_t* vf = a.vt + kvh * DH * a.Sp;

  auto issue = [&](int t) {
    uint4* stage = sm + (t % STAGES) * SCH;
    const int k0 = t * KT;
#pragma unroll
    for (int i = 0; i < IPW; ++i) {
      const int q = wid * IPW + i;
      const int pos = q * 64 + lane;
      const void* src = g_attn_zero;
      if (q * 64 < KCH) {  // K chunk: slot pos -> key row, chunk column
        const int key = pos / KC, slot = pos % KC;
        const int c = slot ^ (key & (KC - 1));
        const int j = k0 + key;
        if (j < P) src = kc + (size_t)j * DH + c * 8;
        else if (j < nkeys) src = kf + (size_t)(j - P) * DH + c * 8;
      } else {             // V^T chunk: slot -> dimension row, 8-key chunk
        const int p2 = pos - KCH;
        const int d = p2 >> 3, slot = p2 & 7;
        const int c = slot ^ (d & 7);
        const int j = k0 + c * 8;
        if (j < P) src = vc + (size_t)d * a.Pc + j;
        else if (j < nkeys) src = vf + (size_t)d * a.Sp + (j - P);
      }
      dma16(src, stage + q * 64);
    }
  };

  f32x4_t o[DH / 16];
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) o[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY, l = 0.f;

#pragma unroll
  for (int st = 0; st < STAGES - 1; ++st)
    if (st < ntiles) issue(st);
  for (int t = 0; t < ntiles; ++t) {
    const int pending = min(STAGES - 2, ntiles - 1 - t);
    if (STAGES >= 3 && pending >= 1) attn_wait_vmcnt<(STAGES >= 3 ? IPW : 0)>();
    else attn_wait_vmcnt<0>();
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    if (t + STAGES - 1 < ntiles) issue(t + STAGES - 1);
    const uint4* sK = sm + (t % STAGES) * SCH;
    const uint4* sV = sK + KCH;
    const int k0 = t * KT;

    // S^T = K Q^T: lane holds keys 16 kt + 4 lg + r of query lq
    f32x4_t sc[KT / 16];
#pragma unroll
    for (int kt = 0; kt < KT / 16; ++kt) {
      sc[kt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      const int row = 16 * kt + lq;
#pragma unroll
      for (int ks = 0; ks < DH / 32; ++ks) {
        const int c = 4 * ks + lg;
        sc[kt] = mfma16a(__builtin_bit_cast(bf16x8_t, sK[row * KC + (c ^ (row & (KC - 1)))]), qf[ks], sc[kt]);
      }
    }
    float tmax = -INFINITY;
    const bool tail = k0 + KT > nkeys;  // only the last tile holds keys past the end
#pragma unroll
    for (int kt = 0; kt < KT / 16; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = k0 + 16 * kt + 4 * lg + r;
        const float v = (!tail || key < nkeys) ? sc[kt][r] * a.scale_log2 : -INFINITY;
        sc[kt][r] = v;
        tmax = fmaxf(tmax, v);
      }
    // the four lane groups holding one query's keys: lanes l, l^16, l^32, l^48
    tmax = xor_lanes16(tmax, [](float x, float y) { return fmaxf(x, y); });
    tmax = xor_lanes32(tmax, [](float x, float y) { return fmaxf(x, y); });
    const float mn = fmaxf(m, tmax);  // finite: every tile holds at least one key
    const float alpha = __builtin_amdgcn_exp2f(m - mn);
    float psum = 0.f;
#pragma unroll
    for (int kt = 0; kt < KT / 16; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float pv = __builtin_amdgcn_exp2f(sc[kt][r] - mn);
        sc[kt][r] = pv;
        psum += pv;
      }
    psum = xor_lanes16(psum, [](float x, float y) { return x + y; });
    psum = xor_lanes32(psum, [](float x, float y) { return x + y; });
    l = l * alpha + psum;
    m = mn;
#pragma unroll
    for (int dt = 0; dt < DH / 16; ++dt) o[dt] *= alpha;

    // O^T += V^T P^T over two 32-key steps; slot order: keys 32 s2 + 4 lg + {0..3}, then +16
#pragma unroll
    for (int s2 = 0; s2 < KT / 32; ++s2) {
      uint32_t hi[4], lo[4];
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        const float p0 = sc[2 * s2 + (x >> 1)][(x & 1) * 2], p1 = sc[2 * s2 + (x >> 1)][(x & 1) * 2 + 1];
        hi[x] = f2bf2(p0, p1);
        lo[x] = f2bf2(p0 - __uint_as_float(hi[x] << 16), p1 - __uint_as_float(hi[x] & 0xFFFF0000u));
      }
      const bf16x8_t phi = __builtin_bit_cast(bf16x8_t, make_uint4(hi[0], hi[1], hi[2], hi[3]));
      const bf16x8_t plo = __builtin_bit_cast(bf16x8_t, make_uint4(lo[0], lo[1], lo[2], lo[3]));
      const int c0 = 4 * s2 + (lg >> 1), c1 = c0 + 2, half = lg & 1;
#pragma unroll
      for (int dt = 0; dt < DH / 16; ++dt) {
        const int d = 16 * dt + lq;
        const uint2* r0 = reinterpret_cast<const uint2*>(sV + d * 8 + (c0 ^ (d & 7))) + half;
        const uint2* r1 = reinterpret_cast<const uint2*>(sV + d * 8 + (c1 ^ (d & 7))) + half;
        const uint2 v0 = *r0, v1 = *r1;
        const bf16x8_t va = __builtin_bit_cast(bf16x8_t, make_uint4(v0.x, v0.y, v1.x, v1.y));
        o[dt] = mfma16a(va, phi, o[dt]);
        o[dt] = mfma16a(va, plo, o[dt]);
      }
    }
  }

  if (qrow < S) {
    const float inv = 1.0f / l;
    bf16_t* dst = a.o + (((size_t)b * S + qrow) * a.H + h) * DH + 4 * lg;
#pragma unroll
    for (int dt = 0; dt < DH / 16; ++dt) {
      uint2 w;
      w.x = f2bf2(o[dt][0] * inv, o[dt][1] * inv);
      w.y = f2bf2(o[dt][2] * inv, o[dt][3] * inv);
      *reinterpret_cast<uint2*>(dst + 16 * dt) = w;
    }
  }
}

template <int NW, int STAGES>
static void run_attn(const AttnArgs& a, hipStream_t s) {
  const int units = ((a.S + 16 * NW - 1) / (16 * NW)) * a.H * a.B;
  dim3 grid(8 * ((units + 7) / 8));
  const size_t lds = (size_t)STAGES * (KT * (a.dh / 8) + a.dh * (KT / 8)) * 16;
  if (a.dh == 128) {
    auto kern = attn_kernel<NW, 128, STAGES>;
    static bool set = false;
    if (!set) {
      (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      set = true;
    }
    hipLaunchKernelGGL(kern, grid, dim3(NW * 64), lds, s, a);
  } else {
    auto kern = attn_kernel<NW, 64, STAGES>;
    static bool set = false;
    if (!set) {
      (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      set = true;
    }
    hipLaunchKernelGGL(kern, grid, dim3(NW * 64), lds, s, a);
  }
}

// A two-stage ring; 64 queries (4 waves) per workgroup for short blocks, 128 (8 waves) from 512
// queries up, where eight waves share each key/value tile: measured on MI355X, 8 waves take 91 us
// instead of 112 us for Dream-7B at 4 x 768 tokens and 95 instead of 104 us for LLaDA-8B at 1280,
// while 4 waves stay best at 384 tokens and for 64-token blocks over a cached prefix.
void launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.S >= 512) run_attn<8, 2>(a, s);
  else run_attn<4, 2>(a, s);
}

// ---------------------------------------------------------------- cache write-back
// One thread per 16-byte key chunk, then one per value element (the value rows are key-contiguous
// and the write offset P + s need not be 8-aligned at a ragged S).
__global__ void __launch_bounds__(256) kv_writeback_kernel(const bf16_t* __restrict__ k, const bf16_t* __restrict__ vt,
                                                          bf16_t* __restrict__ kc, bf16_t* __restrict__ vc, int BH,
                                                          int S, int Sp, int dh, int P, int Pc) {
  const size_t nk = (size_t)BH * S * (dh / 8), nv = (size_t)BH * dh * S;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < nk + nv; i += (size_t)gridDim.x * blockDim.x) {
    if (i < nk) {
      const size_t c = i % (dh / 8), rest = i / (dh / 8);
      const size_t s = rest % S, bh = rest / S;
      *reinterpret_cast<uint4*>(kc + (bh * Pc + P + s) * dh + 8 * c) =
          *reinterpret_cast<const uint4*>(k + (bh * S + s) * dh + 8 * c);
    } else {
      const size_t e = i - nk;
      const size_t s = e % S, rest = e / S;  // rest = bh * dh + d
      vc[rest * Pc + P + s] = vt[rest * Sp + s];
    }
  }
}

void launch_kv_writeback(const bf16_t* k, const bf16_t* vt, bf16_t* kc, bf16_t* vc, int B, int Hkv, int S, int Sp,
                         int dh, int P, int Pc, hipStream_t s) {
  const size_t n = (size_t)B * Hkv * S * (dh / 8 + dh);
  if (n == 0) return;
  const int grid = (int)((n + 255) / 256 < 8 * 1024 ? (n + 255) / 256 : 8 * 1024);
  hipLaunchKernelGGL(kv_writeback_kernel, dim3(grid), dim3(256), 0, s, k, vt, kc, vc, B * Hkv, S, Sp, dh, P, Pc);
}


}  // namespace dcl
