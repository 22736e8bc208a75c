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

__device__ __forceinline__ f32x4_t mfma16a(const bf16x8_t& a, const bf16x8_t& b, const f32x4_t& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

template <int NW, int DH>
__global__ void __launch_bounds__(NW * 64) attn_kernel(AttnArgs a) {
  constexpr int BQ = 16 * NW, NT = NW * 64;
  constexpr int KP = DH + 8;  // padded K row (keys x dims)
  constexpr int VP = KT + 8;  // padded V^T row (dims x keys)
  __shared__ __attribute__((aligned(16))) bf16_t sK[KT * KP];
  __shared__ __attribute__((aligned(16))) bf16_t sV[DH * VP];

  const int qt = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int g = h / (a.H / a.Hkv);
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int lq = lane & 15, lg = lane >> 4;
  const int S = a.S, P = a.P, nkeys = P + S;
  const int qrow = qt * BQ + wid * 16 + lq;

  // Q fragments (B operand): query lq, dims [32 ks + 8 lg, +8)
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
  const bf16_t* kc = a.kc ? a.kc + kvh * P * DH : nullptr;
  const bf16_t* kf = a.k + kvh * S * DH;
  const bf16_t* vc = a.vc ? a.vc + kvh * DH * P : nullptr;
  const bf16_t* vf = a.vt + kvh * DH * a.Sp;

  f32x4_t o[DH / 16];
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) o[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY, l = 0.f;

  for (int k0 = 0; k0 < nkeys; k0 += KT) {
    // K tile [KT keys][DH]
#pragma unroll
    for (int c = tid; c < KT * DH / 8; c += NT) {
      const int key = c / (DH / 8), col = (c % (DH / 8)) * 8, j = k0 + key;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (j < P) v = *reinterpret_cast<const uint4*>(kc + (size_t)j * DH + col);
      else if (j < nkeys) v = *reinterpret_cast<const uint4*>(kf + (size_t)(j - P) * DH + col);
      *reinterpret_cast<uint4*>(sK + key * KP + col) = v;
    }
    // V^T tile [DH][KT keys]; P % 8 == 0 and Sp % 8 == 0 keep every full 8-key chunk in one source
#pragma unroll
    for (int c = tid; c < DH * KT / 8; c += NT) {
      const int d = c / (KT / 8), kk = (c % (KT / 8)) * 8, j = k0 + kk;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (j + 8 <= nkeys) {
        v = (j < P) ? *reinterpret_cast<const uint4*>(vc + (size_t)d * P + j)
                    : *reinterpret_cast<const uint4*>(vf + (size_t)d * a.Sp + (j - P));
      } else if (j < nkeys) {
        uint16_t e[8];
#pragma unroll
        for (int x = 0; x < 8; ++x) {
          const int jj = j + x;
          e[x] = jj >= nkeys ? 0 : (jj < P ? vc[(size_t)d * P + jj] : vf[(size_t)d * a.Sp + (jj - P)]);
        }
        v = make_uint4(e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16), e[6] | (e[7] << 16));
      }
      *reinterpret_cast<uint4*>(sV + d * VP + kk) = v;
    }
    __syncthreads();

    // S^T = K Q^T: lane holds keys 16 kt + 4 lg + r of query lq
    f32x4_t sc[KT / 16];
#pragma unroll
    for (int kt = 0; kt < KT / 16; ++kt) {
      sc[kt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      const bf16_t* kp = sK + (16 * kt + lq) * KP + 8 * lg;
#pragma unroll
      for (int ks = 0; ks < DH / 32; ++ks)
        sc[kt] = mfma16a(*reinterpret_cast<const bf16x8_t*>(kp + 32 * ks), qf[ks], sc[kt]);
    }
    float tmax = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < KT / 16; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = k0 + 16 * kt + 4 * lg + r;
        const float v = key < nkeys ? sc[kt][r] * a.scale_log2 : -INFINITY;
        sc[kt][r] = v;
        tmax = fmaxf(tmax, v);
      }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float mn = fmaxf(m, tmax);
    const float alpha = exp2f(m - mn);
    float psum = 0.f;
#pragma unroll
    for (int kt = 0; kt < KT / 16; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float pv = exp2f(sc[kt][r] - mn);
        sc[kt][r] = pv;
        psum += pv;
      }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
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
        const bf16_t h0 = f2bf(p0), h1 = f2bf(p1);
        hi[x] = (uint32_t)h0 | ((uint32_t)h1 << 16);
        lo[x] = (uint32_t)f2bf(p0 - bf2f(h0)) | ((uint32_t)f2bf(p1 - bf2f(h1)) << 16);
      }
      const bf16x8_t phi = __builtin_bit_cast(bf16x8_t, make_uint4(hi[0], hi[1], hi[2], hi[3]));
      const bf16x8_t plo = __builtin_bit_cast(bf16x8_t, make_uint4(lo[0], lo[1], lo[2], lo[3]));
#pragma unroll
      for (int dt = 0; dt < DH / 16; ++dt) {
        const bf16_t* vp = sV + (16 * dt + lq) * VP + 32 * s2 + 4 * lg;
        const uint2 v0 = *reinterpret_cast<const uint2*>(vp);
        const uint2 v1 = *reinterpret_cast<const uint2*>(vp + 16);
        const bf16x8_t va = __builtin_bit_cast(bf16x8_t, make_uint4(v0.x, v0.y, v1.x, v1.y));
        o[dt] = mfma16a(va, phi, o[dt]);
        o[dt] = mfma16a(va, plo, o[dt]);
      }
    }
    __syncthreads();
  }

  if (qrow < S) {
    const float inv = 1.0f / l;
    bf16_t* dst = a.o + (((size_t)b * S + qrow) * a.H + h) * DH + 4 * lg;
#pragma unroll
    for (int dt = 0; dt < DH / 16; ++dt) {
      uint2 w;
      w.x = (uint32_t)f2bf(o[dt][0] * inv) | ((uint32_t)f2bf(o[dt][1] * inv) << 16);
      w.y = (uint32_t)f2bf(o[dt][2] * inv) | ((uint32_t)f2bf(o[dt][3] * inv) << 16);
      *reinterpret_cast<uint2*>(dst + 16 * dt) = w;
    }
  }
}

template <int NW>
static void run_attn(const AttnArgs& a, hipStream_t s) {
  dim3 grid((a.S + 16 * NW - 1) / (16 * NW), a.H, a.B);
  if (a.dh == 128)
    hipLaunchKernelGGL((attn_kernel<NW, 128>), grid, dim3(NW * 64), 0, s, a);
  else
    hipLaunchKernelGGL((attn_kernel<NW, 64>), grid, dim3(NW * 64), 0, s, a);
}

void launch_attention(const AttnArgs& a, hipStream_t s) {
  const long blocks4 = (long)((a.S + 63) / 64) * a.H * a.B;
  if (blocks4 >= 512)
    run_attn<4>(a, s);
  else
    run_attn<2>(a, s);
}

}  // namespace dcl
