// Non-causal (bidirectional) flash-style attention for gfx950, MHA and GQA, head_dim 64 / 128.
//
// Masked diffusion LMs attend from every position to every position; there is no causal mask, so
// the whole S x S score matrix is real work. One workgroup handles 16*NQ queries of one (batch,
// head); each wavefront owns 16 queries and walks its share of the keys in tiles of KT (32 or 64)
// with an online softmax in float32. Keys are [cached prefix (P) || the S fresh tokens].
//
// Orientation: the score tile is computed transposed, S^T = K Q^T (MFMA A = K from LDS, B = Q held
// in registers), so each lane holds 16 scores of ONE query. Its softmax probabilities then feed the
// P*V product directly as the MFMA B operand of O^T = V^T P^T, with V^T read from a key-contiguous
// LDS tile in the matching key order; no register shuffle of P is needed.
// P is split into three bf16 parts (hi + mid + lo, three MFMAs), so the probabilities enter the
// product with at least 24 significant bits, as in a float32 evaluation. Two parts (16 bits) were
// measurably less accurate than float32: on sequences of 5-8 tokens they flipped the bf16 rounding
// of about a quarter of the final hidden states of a small model against a float64 reference.
#include <type_traits>

#include "dcl_internal.h"

namespace dcl {



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
// Wait until all but this wave's `newer` most recently issued stages (IPW loads each) landed.
template <int IPW, int MAXN>
__device__ __forceinline__ void attn_wait_stages(int newer) {
  if constexpr (MAXN > 0) {
    static_assert(MAXN * IPW < 64, "vmcnt range");
    if (newer >= MAXN) {
      attn_wait_vmcnt<MAXN * IPW>();
      return;
    }
    attn_wait_stages<IPW, MAXN - 1>(newer);
  } else {
    attn_wait_vmcnt<0>();
  }
}

// K and V^T tiles move HBM/L2 -> LDS with global_load_lds_dwordx4 into a STAGES-deep ring (no
// register staging, no padding). K rows (DH/8 chunks of 16 bytes) are XOR-swizzled by the key
// index, V^T rows (KT/8 chunks of 8 keys) by the dimension index. Both are read in whole 16-byte
// chunks, bank-conflict free; the V^T fragments are then assembled by a lane-row swap (below).
// Chunks past the last key repeat real data (see below).
//
// Key groups: the NQ * KG waves of a workgroup are NQ query waves (16 queries each) times KG key
// groups. Step t of the ring holds the KG key tiles t*KG .. t*KG + KG - 1; key group g works on
// tile t*KG + g, so each wave's serial chain (scores -> softmax -> P V) covers 1/KG of the keys
// and KG times as many waves hide each other's latencies. At the end the groups' running
// (max, sum, unnormalised output) are combined through LDS in group order, which keeps the result
// independent of timing.
template <int NQ, int KG, int KT, int DH, int STAGES>
__global__ void __launch_bounds__(NQ * KG * 64) attn_kernel(AttnArgs a) {
  constexpr int BQ = 16 * NQ, NWAVE = NQ * KG;
  constexpr int KC = DH / 8;           // chunks per K row
  constexpr int VC = KT / 8;           // chunks per V^T row
  constexpr int KCH = KT * KC;         // K chunks per tile
  constexpr int VCH = DH * VC;         // V^T chunks per tile
  constexpr int TCH = KCH + VCH;       // chunks per tile
  constexpr int SCH = KG * TCH;        // chunks per ring step
  constexpr int IPW = SCH / 64 / NWAVE;  // load instructions per wave per ring step
  static_assert((KT == 32 || KT == 64) && SCH % (64 * NWAVE) == 0 && KCH % 64 == 0 && VCH % 64 == 0 &&
                    STAGES >= 2 && IPW * (STAGES - 2) < 64 && NWAVE <= 16,
                "stage shape");
  static_assert(KG == 1 || (size_t)(KG - 1) * NQ * (DH / 16) * 64 * 16 + (size_t)(KG - 1) * NQ * 64 * 8 <=
                                (size_t)STAGES * SCH * 16,
                "the group merge reuses the ring");
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
  const int tid = threadIdx.x, lane = tid & 63, wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qw = wid % NQ, kg = wid / NQ;
  const int lq = lane & 15, lg = lane >> 4;
  const int S = a.S, P = a.P, Sk = a.Sk ? a.Sk : a.S, nkeys = P + Sk;  // S queries; P cached + Sk fresh keys
  const int qrow = qt * BQ + qw * 16 + lq;
  const int ntiles = (nkeys + KT - 1) / KT;
  const int nsteps = (ntiles + KG - 1) / KG;

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
  const bf16_t* kf = a.k + kvh * Sk * DH;
  const bf16_t* vc = a.vc ? a.vc + kvh * DH * a.Pc : nullptr;
  const bf16_t* vf = a.vt + kvh * DH * a.Sp;

  f32x4_t o[DH / 16];
#pragma unroll
  for (int dt = 0; dt < DH / 16; ++dt) o[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // per query: reference point m (log2 units, scaled; within 2^8 of the running maximum, see the
  // lazy rescaling below) and the sum l of exp2(score - m)
  float m = -INFINITY, l = 0.f;
  const float scale = a.scale_log2;

  // DMA assignment: instruction i of wave w fills the 64-chunk block b = i * NWAVE + w of a ring
  // step (block sizes are multiples of NWAVE, so the key group and the K / V^T role of instruction i
  // are compile-time). Per ring step only the tile origin k0 changes: a chunk at key j < P comes
  // from the cache, j < P + Sk from the fresh keys/values. A chunk past the last key re-reads the
  // last key's (or last 8-key chunk's) data: those keys score -inf, so their probability is
  // exactly 0 against finite values, and the address stays branch-free.
  static_assert((KCH / 64) % NWAVE == 0 && (VCH / 64) % NWAVE == 0, "DMA blocks per wave");
  constexpr int TB = TCH / 64;  // 64-chunk blocks per key tile
  int jrel[IPW], offc[IPW];
  const bf16_t* fsrc[IPW];  // fresh-key source for the tile origin k0 = P
#pragma unroll
  for (int i = 0; i < IPW; ++i) {
    const int bb = (i * NWAVE) % TB;       // block within the key tile (same for every wave's lane 0)
    const int pos = (bb + wid) * 64 + lane;  // chunk within the key tile
    if ((i * NWAVE) % TB < KCH / 64) {     // K chunk: slot pos -> key row, chunk column
      const int key = pos / KC, c = (pos % KC) ^ (key & (KC - 1));
      jrel[i] = key;
      offc[i] = key * DH + c * 8;
      fsrc[i] = kf + key * DH + c * 8;
    } else {                                // V^T chunk: slot -> dimension row, 8-key chunk
      const int p2 = pos - KCH;
      const int d = p2 / VC, c = (p2 % VC) ^ (d & (VC - 1));
      jrel[i] = c * 8;
      offc[i] = d * a.Pc + c * 8;
      fsrc[i] = vf + (size_t)d * a.Sp + c * 8;
    }
  }
  const uint32_t lds_base = lds_addr_of(sm) + (uint32_t)wid * 1024u;
  const int klast = nkeys - 1, vlast = (nkeys - 1) & ~7;  // last key, start of the last 8-key chunk
  const int vlast_f = (Sk - 1) & ~7;                         // the same for the fresh values alone
  // the main loop below is instantiated twice: without (kFresh) and with a cached prefix
  auto main_loop = [&](auto fresh_only) {
    constexpr bool kFresh = decltype(fresh_only)::value;
    auto issue = [&](int t) {
      const uint32_t stage = lds_base + (uint32_t)((t % STAGES) * SCH) * 16u;
#pragma unroll
      for (int i = 0; i < IPW; ++i) {
        const bool isk = (i * NWAVE) % TB < KCH / 64;
        const int mult = isk ? DH : 1;
        const int k0 = (t * KG + (i * NWAVE) / TB) * KT;
        const int j = k0 + jrel[i];
        const void* src;
        if constexpr (kFresh) {
          const int jc = min(j, isk ? klast : vlast);
          src = fsrc[i] + (ptrdiff_t)(jc - jrel[i]) * mult;
        } else {
          // fresh side with the same clamping as above, in fresh-key indices; the cache side holds
          // keys j < P (P is a multiple of 8, so no 8-key chunk straddles the two)
          const int jf = min(j - P, isk ? klast - P : vlast_f);
          const bf16_t* fp = fsrc[i] + (ptrdiff_t)(jf - jrel[i]) * mult;
          const bf16_t* cp = (isk ? kc : vc) + offc[i] + (ptrdiff_t)k0 * mult;
          src = j < P ? cp : fp;
        }
        dma16_at(src, stage + (uint32_t)(i * NWAVE) * 1024u);
      }
    };

#pragma unroll
    for (int st = 0; st < STAGES - 1; ++st)
      if (st < nsteps) issue(st);
    for (int t = 0; t < nsteps; ++t) {
      // step t landed; the steps t + 1 .. min(nsteps - 1, t + STAGES - 2) may still fly
      attn_wait_stages<IPW, STAGES - 2>(min(STAGES - 2, nsteps - 1 - t));
      asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
      if (t + STAGES - 1 < nsteps) issue(t + STAGES - 1);
      const int k0 = (t * KG + kg) * KT;
      if (k0 >= nkeys) continue;  // this group's tile is past the end (uniform per wave)
      const uint4* sK = sm + (t % STAGES) * SCH + kg * TCH;
      const uint4* sV = sK + KCH;

      // S^T = K Q^T: lane holds keys 16 kt + 4 lg + r of query lq. The tile's K fragments are read
      // first and the independent accumulation chains interleaved.
      bf16x8_t kfr[KT / 16][DH / 32];
#pragma unroll
      for (int kt = 0; kt < KT / 16; ++kt) {
        const int row = 16 * kt + lq;
#pragma unroll
        for (int ks = 0; ks < DH / 32; ++ks) {
          const int c = 4 * ks + lg;
          kfr[kt][ks] = __builtin_bit_cast(bf16x8_t, sK[row * KC + (c ^ (row & (KC - 1)))]);
        }
      }
      f32x4_t sc[KT / 16];
#pragma unroll
      for (int kt = 0; kt < KT / 16; ++kt) sc[kt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < DH / 32; ++ks)
#pragma unroll
        for (int kt = 0; kt < KT / 16; ++kt) sc[kt] = mfma16a(kfr[kt][ks], qf[ks], sc[kt]);
      // V^T fragments, read while the softmax below runs: dimension 16 dt + lq at the keys
      // 32 s2 + 4 lg + {0..3} and 32 s2 + 16 + 4 lg + {0..3} (the order in which the score MFMA left
      // the probabilities in the lanes). Each lane reads one whole 16-byte chunk (bank-conflict free
      // through the XOR swizzle, as the K reads): lane groups 0 / 1 / 2 / 3 read the keys
      // 0-7 / 16-23 / 8-15 / 24-31 of the 32-key block, and neighbouring groups (0, 1) and (2, 3)
      // exchange halves with v_permlane16_swap, which swaps the odd 16-lane rows of its first operand
      // with the even rows of its second: group 0 keeps keys 0-3 and receives 16-19, group 1 receives
      // 4-7 and keeps 20-23, and likewise for groups 2 and 3.
      bf16x8_t vfr[KT / 32][DH / 16];
#pragma unroll
      for (int s2 = 0; s2 < KT / 32; ++s2) {
        const int cx = 4 * s2 + (((lg & 1) << 1) | (lg >> 1));
#pragma unroll
        for (int dt = 0; dt < DH / 16; ++dt) {
          const int d = 16 * dt + lq;
          const uint4 x = sV[d * VC + (cx ^ (d & (VC - 1)))];
          const auto s0 = __builtin_amdgcn_permlane16_swap(x.x, x.z, false, false);
          const auto s1 = __builtin_amdgcn_permlane16_swap(x.y, x.w, false, false);
          vfr[s2][dt] = __builtin_bit_cast(bf16x8_t, make_uint4(s0[0], s1[0], s0[1], s1[1]));
        }
      }
      if (k0 + KT > nkeys) {  // only the last tile holds keys past the end
#pragma unroll
        for (int kt = 0; kt < KT / 16; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (k0 + 16 * kt + 4 * lg + r >= nkeys) sc[kt][r] = -INFINITY;
      }
      float tmax = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < KT / 16; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) tmax = fmaxf(tmax, sc[kt][r]);
      // the four lane groups holding one query's keys: lanes l, l^16, l^32, l^48
      tmax = xor_lanes16(tmax, [](float x, float y) { return fmaxf(x, y); });
      tmax = xor_lanes32(tmax, [](float x, float y) { return fmaxf(x, y); });
      // Lazy rescaling: the reference point m only moves when a score exceeds it by more than
      // 2^8 (probabilities up to 256 are exact to represent and sum in float32); the division by
      // the running sum at the end makes the result independent of the reference point. When no
      // lane of the wave moves, the output rescale is skipped.
      const float ts = tmax * scale;
      const bool move = ts > m + 8.f;  // true on the first processed tile (m = -inf)
      const float mn = move ? ts : m;
      float psum = 0.f;
#pragma unroll
      for (int kt = 0; kt < KT / 16; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float pv = __builtin_amdgcn_exp2f(fmaf(sc[kt][r], scale, -mn));
          sc[kt][r] = pv;
          psum += pv;
        }
      psum = xor_lanes16(psum, [](float x, float y) { return x + y; });
      psum = xor_lanes32(psum, [](float x, float y) { return x + y; });
      if (__builtin_amdgcn_ballot_w64(move)) {
        const float alpha = __builtin_amdgcn_exp2f(m - mn);  // 1 in the lanes that keep m
        l *= alpha;
#pragma unroll
        for (int dt = 0; dt < DH / 16; ++dt) o[dt] *= alpha;
      }
      l += psum;
      m = mn;

      // O^T += V^T P^T over 32-key steps; P enters as three bf16 parts (hi + mid + lo)
#pragma unroll
      for (int s2 = 0; s2 < KT / 32; ++s2) {
        uint32_t hi[4], mi[4], lo[4];
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          const float p0 = sc[2 * s2 + (x >> 1)][(x & 1) * 2], p1 = sc[2 * s2 + (x >> 1)][(x & 1) * 2 + 1];
          hi[x] = f2bf2(p0, p1);
          const float r0 = p0 - __uint_as_float(hi[x] << 16), r1 = p1 - __uint_as_float(hi[x] & 0xFFFF0000u);
          mi[x] = f2bf2(r0, r1);
          lo[x] = f2bf2(r0 - __uint_as_float(mi[x] << 16), r1 - __uint_as_float(mi[x] & 0xFFFF0000u));
        }
        const bf16x8_t phi = __builtin_bit_cast(bf16x8_t, make_uint4(hi[0], hi[1], hi[2], hi[3]));
        const bf16x8_t pmi = __builtin_bit_cast(bf16x8_t, make_uint4(mi[0], mi[1], mi[2], mi[3]));
        const bf16x8_t plo = __builtin_bit_cast(bf16x8_t, make_uint4(lo[0], lo[1], lo[2], lo[3]));
#pragma unroll
        for (int dt = 0; dt < DH / 16; ++dt) o[dt] = mfma16a(vfr[s2][dt], phi, o[dt]);
#pragma unroll
        for (int dt = 0; dt < DH / 16; ++dt) o[dt] = mfma16a(vfr[s2][dt], pmi, o[dt]);
#pragma unroll
        for (int dt = 0; dt < DH / 16; ++dt) o[dt] = mfma16a(vfr[s2][dt], plo, o[dt]);
      }
    }

  };
  if (P == 0) main_loop(std::integral_constant<bool, true>{});
  else main_loop(std::integral_constant<bool, false>{});

  if constexpr (KG > 1) {
    // groups 1 .. KG-1 park (m, l, o) in the ring; group 0 folds them in group order
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    f32x4_t* xo = reinterpret_cast<f32x4_t*>(sm);
    float2* xml = reinterpret_cast<float2*>(xo + (size_t)(KG - 1) * NQ * (DH / 16) * 64);
    if (kg > 0) {
      const int base = (kg - 1) * NQ + qw;
#pragma unroll
      for (int dt = 0; dt < DH / 16; ++dt) xo[((size_t)base * (DH / 16) + dt) * 64 + lane] = o[dt];
      xml[base * 64 + lane] = make_float2(m, l);
    }
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    if (kg > 0) return;
#pragma unroll
    for (int gg = 1; gg < KG; ++gg) {
      const int base = (gg - 1) * NQ + qw;
      const float2 ml = xml[base * 64 + lane];
      if (ml.x == -INFINITY) continue;  // a group that saw no key
      const float mn = fmaxf(m, ml.x);
      const float ea = __builtin_amdgcn_exp2f(m - mn), eb = __builtin_amdgcn_exp2f(ml.x - mn);
      l = l * ea + ml.y * eb;
#pragma unroll
      for (int dt = 0; dt < DH / 16; ++dt) o[dt] = o[dt] * ea + xo[((size_t)base * (DH / 16) + dt) * 64 + lane] * eb;
      m = mn;
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

template <int NQ, int KG, int KT, int STAGES>
static void run_attn(const AttnArgs& a, hipStream_t s) {
  static_assert((size_t)STAGES * KG * (KT * 16 + 128 * (KT / 8)) * 16 <= 160 * 1024, "ring exceeds the LDS of a CU");
  const int units = ((a.S + 16 * NQ - 1) / (16 * NQ)) * a.H * a.B;
  if (units == 0) return;
  dim3 grid(8 * ((units + 7) / 8));
  const size_t lds = (size_t)STAGES * KG * (KT * (a.dh / 8) + a.dh * (KT / 8)) * 16;
  if (a.dh == 128) {
    auto kern = attn_kernel<NQ, KG, KT, 128, STAGES>;
    static std::atomic<uint32_t> lds_set{0};
    ensure_dynamic_lds(reinterpret_cast<const void*>(kern), lds, lds_set);
    hipLaunchKernelGGL(kern, grid, dim3(NQ * KG * 64), lds, s, a);
  } else if constexpr ((KT * 8 / 64) % (NQ * KG) != 0 || (64 * (KT / 8) / 64) % (NQ * KG) != 0) {
    run_attn<4, 2, 64, 2>(a, s);  // this wave layout does not tile head_dim 64: the default one does
  } else {
    auto kern = attn_kernel<NQ, KG, KT, 64, STAGES>;
    static std::atomic<uint32_t> lds_set{0};
    ensure_dynamic_lds(reinterpret_cast<const void*>(kern), lds, lds_set);
    hipLaunchKernelGGL(kern, grid, dim3(NQ * KG * 64), lds, s, a);
  }
}

// A two-stage ring of 32-key tiles: 64 KB of LDS for head_dim 128, so two workgroups share a CU. Few query
// waves (B * H * S / 16 below 4096): 4 query waves x 2 key groups per workgroup, so each wave walks half
// the keys and twice as many waves share a CU; many query waves: 8 query waves x 1 group. Measured on
// MI355X (LLaDA-8B / Dream-7B heads, three-part P), per launch, against the same layouts with 64-key
// tiles (128 KB rings, one workgroup per CU): 384 tokens 12.2 us (12.1), 1280 tokens 73.0 us (87.0),
// 8 x 64 tokens over a 1216-key cache 34.1 us (35.1), Dream-7B 4 x 768 tokens 88.4 us (95.8).
// head_dim 64 falls back to 64-key tiles (a 32-key tile has too few 64-chunk blocks for 8 waves).
void launch_attention(const AttnArgs& a, hipStream_t s) {
  const long query_waves = (long)a.B * a.H * ((a.S + 15) / 16);
  if (query_waves >= 4096) run_attn<8, 1, 32, 2>(a, s);
  else run_attn<4, 2, 32, 2>(a, s);
}

// ---------------------------------------------------------------- cache write-back
// One thread per 16-byte key chunk, then one per value element (the value rows are key-contiguous
// and the write offset P + s need not be 8-aligned). Token s of the step sits in slot koff + s of the
// fresh buffers (k rows of Sk keys, v^T rows of pitch Sp).
__global__ void __launch_bounds__(256) kv_writeback_kernel(const bf16_t* __restrict__ k, const bf16_t* __restrict__ vt,
                                                          bf16_t* __restrict__ kc, bf16_t* __restrict__ vc, int BH,
                                                          int S, int Sk, int Sp, int koff, int dh, int P, int Pc) {
  const size_t nk = (size_t)BH * S * (dh / 8), nv = (size_t)BH * dh * S;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < nk + nv; i += (size_t)gridDim.x * blockDim.x) {
    if (i < nk) {
      const size_t c = i % (dh / 8), rest = i / (dh / 8);
      const size_t s = rest % S, bh = rest / S;
      *reinterpret_cast<uint4*>(kc + (bh * Pc + P + s) * dh + 8 * c) =
          *reinterpret_cast<const uint4*>(k + (bh * Sk + koff + s) * dh + 8 * c);
    } else {
      const size_t e = i - nk;
      const size_t s = e % S, rest = e / S;  // rest = bh * dh + d
      vc[rest * Pc + P + s] = vt[rest * Sp + koff + s];
    }
  }
}

void launch_kv_writeback(const bf16_t* k, const bf16_t* vt, bf16_t* kc, bf16_t* vc, int B, int Hkv, int S, int Sk,
                         int Sp, int koff, int dh, int P, int Pc, hipStream_t s) {
  const size_t n = (size_t)B * Hkv * S * (dh / 8 + dh);
  if (n == 0) return;
  const int grid = (int)((n + 255) / 256 < 8 * 1024 ? (n + 255) / 256 : 8 * 1024);
  hipLaunchKernelGGL(kv_writeback_kernel, dim3(grid), dim3(256), 0, s, k, vt, kc, vc, B * Hkv, S, Sk, Sp, koff, dh, P,
                     Pc);
}

// ---------------------------------------------------------------- carried cache keys
// A cached prefix whose length P is not a multiple of 8 ends inside an 8-key chunk. Attention reads the
// cache only in whole chunks, so the koff = P mod 8 newest cached keys (and values) are copied in front
// of the fresh ones: slots [0, koff) of k [BH, Sk, dh] and of every v^T row (pitch Sp). One thread per
// element.
__global__ void __launch_bounds__(256) kv_carry_kernel(const bf16_t* __restrict__ kc, const bf16_t* __restrict__ vc,
                                                      bf16_t* __restrict__ k, bf16_t* __restrict__ vt, int BH, int Sk,
                                                      int Sp, int dh, int P, int Pc, int koff) {
  const size_t n = (size_t)BH * koff * dh;  // as many key elements as value elements
  const size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
  if (i >= 2 * n) return;
  const int P8 = P - koff;
  if (i < n) {
    const size_t d = i % dh, rest = i / dh;
    const size_t j = rest % koff, bh = rest / koff;
    k[(bh * Sk + j) * dh + d] = kc[(bh * Pc + P8 + j) * dh + d];
  } else {
    const size_t e = i - n;
    const size_t j = e % koff, rest = e / koff;  // rest = bh * dh + d
    vt[rest * Sp + j] = vc[rest * Pc + P8 + j];
  }
}

void launch_kv_carry(const bf16_t* kc, const bf16_t* vc, bf16_t* k, bf16_t* vt, int B, int Hkv, int Sk, int Sp,
                     int dh, int P, int Pc, hipStream_t s) {
  const int koff = P % 8;
  if (koff == 0) return;
  const size_t n = 2 * (size_t)B * Hkv * koff * dh;
  hipLaunchKernelGGL(kv_carry_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, kc, vc, k, vt, B * Hkv, Sk,
                     Sp, dh, P, Pc, koff);
}


}  // namespace dcl
