// Decode attention over the ragged compressed KV cache (gfx950).
//
// SGD-KV keeps its compressed cache per KV head, before the heads are repeated
// for GQA (Appendix A.2), so one segment of rows serves the G query heads of
// its group. Decode reads each segment once for all G heads:
//
//   decode_split: each wave owns one chunk of a segment's rows. Logits of the
//     G heads against 16 keys at a time are one 16x16 MFMA (the G query rows
//     padded to 16 form the A operand). The wave keeps an online softmax
//     (running max m and sum s per head, base-2 units) and accumulates P.V in
//     fp32 on the vector ALU (bf16 V rows are widened exactly); the next
//     step's K and V are already in flight. One partial (m, s, o[d]) per head
//     and chunk is written; waves never synchronise with each other.
//   decode_combine: per (sequence, query head), a fixed-order log-sum-exp
//     merge of the chunk partials; out = o/s, lse = (m + log2 s) * ln 2.
//
// Work is a flattened (chunk, segment) grid, so unequal budgets (one head
// with most of the rows, others with few) still spread over the whole chip.
#include "device_common.h"
#include "mfma_frag.h"
#include "sgdkv_internal.h"

namespace sgdkv {

namespace {
constexpr int kWaves = kBlock / 64;

__device__ __forceinline__ void clamp_segment(const DecodeArgs& a, int seg, int64_t& r0, int64_t& r1) {
  const int nseg = a.B * a.Hkv;
  const rsrc_t orr = make_rsrc(a.offsets, (uint64_t)(nseg + 1) * 8);
  r0 = (int64_t)ld64(orr, (uint32_t)seg * 8);
  r1 = (int64_t)ld64(orr, (uint32_t)(seg + 1) * 8);
  r0 = r0 < 0 ? 0 : (r0 > a.total_rows ? a.total_rows : r0);
  r1 = r1 < r0 ? r0 : (r1 > a.total_rows ? a.total_rows : r1);
}
}  // namespace

// Loads of one 16-key step: the K fragments of the MFMA (key lr, k = 32c + 8*lg)
// and this lane's V rows (keys kg + KG*u, columns col0 .. col0+7).
template <typename T, int D>
struct DecodeStep {
  static constexpr int EB = sizeof(T);
  static constexpr int RB = D * EB;
  static constexpr int NC = D / 32;
  static constexpr int LPR = D / 8;        // lanes sharing one value row (8 columns each)
  static constexpr int KG = 64 / LPR;      // key groups per wave
  static constexpr int VPL = 16 / KG;      // value rows per lane per step
  static constexpr int VW = EB == 2 ? 1 : 2;  // 16-byte pieces per 8 columns
  Frag<T> kb[NC];
  u32x4 vv[VPL][VW];
  __device__ __forceinline__ void load(const rsrc_t& kr, const rsrc_t& vr, int64_t k0, int lr, int lgp, int kg,
                                       int col0) {
#pragma unroll
    for (int c = 0; c < NC; ++c) kb[c] = gload_frag<T>(kr, (uint32_t)((k0 + lr) * RB + (32 * c + 8 * lgp) * EB));
#pragma unroll
    for (int u = 0; u < VPL; ++u)
#pragma unroll
      for (int x = 0; x < VW; ++x) vv[u][x] = ld128(vr, (uint32_t)((k0 + kg + KG * u) * RB + col0 * EB + 16 * x));
  }
  __device__ __forceinline__ void value_row(int u, float (&v)[8]) const {
    if constexpr (EB == 2) {
      const u32x4 x = vv[u][0];
      v[0] = bf16_lo(x.x); v[1] = bf16_hi(x.x); v[2] = bf16_lo(x.y); v[3] = bf16_hi(x.y);
      v[4] = bf16_lo(x.z); v[5] = bf16_hi(x.z); v[6] = bf16_lo(x.w); v[7] = bf16_hi(x.w);
    } else {
      const u32x4 x0 = vv[u][0], x1 = vv[u][VW - 1];
      v[0] = __uint_as_float(x0.x); v[1] = __uint_as_float(x0.y); v[2] = __uint_as_float(x0.z);
      v[3] = __uint_as_float(x0.w); v[4] = __uint_as_float(x1.x); v[5] = __uint_as_float(x1.y);
      v[6] = __uint_as_float(x1.z); v[7] = __uint_as_float(x1.w);
    }
  }
};

__device__ __forceinline__ void wave_sync() {
  // order this wave's LDS writes before its following LDS reads (other lanes read them)
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Maximum over the 16 lanes of a row (lanes 16r .. 16r+15), by DPP rotations.
__device__ __forceinline__ float row16_max(float x) {
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x128, 0xF, 0xF, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x124, 0xF, 0xF, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x122, 0xF, 0xF, false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x121, 0xF, 0xF, false)));
  return x;
}
__device__ __forceinline__ float row16_sum(float x) {
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x128, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x124, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x122, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x121, 0xF, 0xF, false));
  return x;
}

// One wave's pass over its chunk. Lane (lr, lg) of the logit MFMA holds key lr
// of the step for heads 4*lg+i. Every head keeps a reference m (base-2 units)
// and the lane-local sums s = sum 2^(y - m) and o = sum 2^(y - m) v.
//   EXACT = false: m is the head's largest logit of the chunk's first step and
//     stays fixed, so a logit costs one fma and one exp2 and nothing rescales.
//     The caller checks the result for overflow and then reruns the chunk
//     with EXACT = true.
//   EXACT = true: m is the running maximum; s and o are rescaled when it moves.
// The probabilities of a step reach the P.V lanes through LDS (double
// buffered by step parity, so one wave-local sync per step orders both the
// writes before the reads and the reads before the writes two steps later).
template <typename T, int D, int GM, int PF, bool EXACT>
__device__ __forceinline__ void decode_chunk(const DecodeArgs& a, float (*pls)[16][16], float (*als)[16],
                                             const rsrc_t& kr, const rsrc_t& vr, int64_t c0, int64_t c1,
                                             const Frag<T> (&qa)[D / 32], int lane, float (&m)[4], float (&s)[4],
                                             float (&o)[GM][8]) {
  using S = DecodeStep<T, D>;
  constexpr int KS = 16;
  constexpr int NBUF = PF + 1;
  const int lr = lane & 15, lgp = lane >> 4;
  const int kg = lane / S::LPR, col0 = 8 * (lane % S::LPR);
  const int G = a.G;
  const float c2 = a.c2;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    m[i] = -INFINITY;
    s[i] = 0.f;
  }
#pragma unroll
  for (int g = 0; g < GM; ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) o[g][e] = 0.f;
  const int nsteps = (int)((c1 - c0 + KS - 1) / KS);
  S buf[NBUF];
#pragma unroll
  for (int p = 0; p < PF; ++p)
    if (p < nsteps) buf[p].load(kr, vr, c0 + p * KS, lr, lgp, kg, col0);
  for (int it0 = 0; it0 < nsteps; it0 += NBUF) {
#pragma unroll
    for (int u = 0; u < NBUF; ++u) {
      const int it = it0 + u;
      if (it >= nsteps) break;
      const int64_t k0 = c0 + (int64_t)it * KS;
      if (it + PF < nsteps) buf[(u + PF) % NBUF].load(kr, vr, k0 + PF * KS, lr, lgp, kg, col0);
      const S& cur = buf[u];
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < S::NC; ++c) acc = mma(qa[c], cur.kb[c], acc);
      const bool valid = k0 + lr < c1;
      float alpha[4] = {1.f, 1.f, 1.f, 1.f};
      if (EXACT || it == 0) {
        // running (or first-step) maximum per head over the 16 keys
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float mx = row16_max(valid ? acc[i] * c2 : -INFINITY);
          const float mn = fmaxf(m[i], mx);
          if (EXACT) alpha[i] = (m[i] == -INFINITY) ? (mn == -INFINITY ? 1.f : 0.f) : fast_exp2(m[i] - mn);
          m[i] = mn;
        }
      }
      float p[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        p[i] = (valid && m[i] != -INFINITY) ? fast_exp2(fmaf(acc[i], c2, -m[i])) : 0.f;
        s[i] = EXACT ? fmaf(s[i], alpha[i], p[i]) : s[i] + p[i];
      }
      float(*pw)[16] = pls[it & 1];
      *reinterpret_cast<f32x4*>(&pw[lr][4 * lgp]) = f32x4{p[0], p[1], p[2], p[3]};
      bool moved = false;
      if (EXACT) {
        if (lr == 0) *reinterpret_cast<f32x4*>(&als[it & 1][4 * lgp]) = f32x4{alpha[0], alpha[1], alpha[2], alpha[3]};
        moved = __any(alpha[0] != 1.f || alpha[1] != 1.f || alpha[2] != 1.f || alpha[3] != 1.f);
      }
      wave_sync();
      if (EXACT && moved) {
#pragma unroll
        for (int g = 0; g < GM; ++g)
          if (g < G) {
            const float al = als[it & 1][g];
#pragma unroll
            for (int e = 0; e < 8; ++e) o[g][e] *= al;
          }
      }
      // P.V for this lane's value rows and columns
#pragma unroll
      for (int u2 = 0; u2 < S::VPL; ++u2) {
        const int kk = kg + S::KG * u2;
        float v[8];
        cur.value_row(u2, v);
        float pk[GM];
#pragma unroll
        for (int g4 = 0; g4 < GM; g4 += 4) {
          const f32x4 q4 = *reinterpret_cast<const f32x4*>(&pw[kk][g4]);
          pk[g4] = q4[0];
          if (g4 + 1 < GM) pk[g4 + 1] = q4[1];
          if (g4 + 2 < GM) pk[g4 + 2] = q4[2];
          if (g4 + 3 < GM) pk[g4 + 3] = q4[3];
        }
#pragma unroll
        for (int g = 0; g < GM; ++g)
          if (g < G) {
#pragma unroll
            for (int e = 0; e < 8; ++e) o[g][e] = fmaf(pk[g], v[e], o[g][e]);
          }
      }
    }
  }
}

// GM = compile-time bound on the group size (8 or 16); PF = steps of K/V in
// flight ahead of the one being computed. Each wave owns one chunk of a
// segment: chunk index = 4*blockIdx.x + wave.
template <typename T, int D, int GM, int PF>
__global__ __launch_bounds__(kBlock, 2) void decode_split_kernel(DecodeArgs a) {
  using S = DecodeStep<T, D>;
  __shared__ __attribute__((aligned(16))) float pls[kWaves][2][16][16];  // probabilities [key][head]
  __shared__ __attribute__((aligned(16))) float als[kWaves][2][16];      // per-head rescale (exact pass)

  const int seg = blockIdx.y;
  const int b = seg / a.Hkv, h = seg % a.Hkv;
  const int tid = threadIdx.x, wid = tid >> 6, lane = tid & 63;
  int64_t r0, r1;
  clamp_segment(a, seg, r0, r1);
  const int64_t len = r1 - r0;
  const int64_t chunk = (int64_t)blockIdx.x * kWaves + wid;
  const int64_t c0 = chunk * a.chunk;
  if (c0 >= len) return;  // this wave's chunk is past the segment (waves never synchronise)
  const int64_t c1 = c0 + a.chunk < len ? c0 + a.chunk : len;

  const int lr = lane & 15, lgp = lane >> 4;
  const int G = a.G;
  const rsrc_t kr = make_rsrc(static_cast<const char*>(a.k_c) + r0 * S::RB, (uint64_t)len * S::RB);
  const rsrc_t vr = make_rsrc(static_cast<const char*>(a.v_c) + r0 * S::RB, (uint64_t)len * S::RB);
  const rsrc_t qr = make_rsrc(static_cast<const char*>(a.q) + ((int64_t)b * a.Hq + (int64_t)h * G) * S::RB,
                              (uint64_t)G * S::RB);
  Frag<T> qa[S::NC];  // row lr = head; rows >= G read as zeros
#pragma unroll
  for (int c = 0; c < S::NC; ++c) qa[c] = gload_frag<T>(qr, (uint32_t)(lr * S::RB + (32 * c + 8 * lgp) * S::EB));

  float m[4], s[4], o[GM][8];
  decode_chunk<T, D, GM, PF, false>(a, pls[wid], als[wid], kr, vr, c0, c1, qa, lane, m, s, o);
  // 2^64 bounds every probability, so s and o stay finite unless V is huge or the
  // first step's maximum sat far below a later logit: then redo with rescaling
  bool bad = false;
#pragma unroll
  for (int i = 0; i < 4; ++i) bad |= !(s[i] <= 1.8446744073709552e19f);
#pragma unroll
  for (int g = 0; g < GM; ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) bad |= !(fabsf(o[g][e]) < INFINITY);
  if (__any(bad)) decode_chunk<T, D, GM, PF, true>(a, pls[wid], als[wid], kr, vr, c0, c1, qa, lane, m, s, o);

  // Reduce within the wave: the 16 lanes of each head's sum, the KG key groups of o.
#pragma unroll
  for (int i = 0; i < 4; ++i) s[i] = row16_sum(s[i]);
#pragma unroll
  for (int g = 0; g < GM; ++g)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float x = o[g][e];
#pragma unroll
      for (int sft = S::LPR; sft < 64; sft <<= 1) x += __shfl_xor(x, sft, 64);
      o[g][e] = x;
    }
  // write this chunk's partial (m, s, o[D]) for each of the G heads
  const int stride = D + 2;
  const int64_t bq0 = (int64_t)b * a.Hq + (int64_t)h * G;
  if (lr == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int hd = 4 * lgp + i;
      if (hd < G) {
        const rsrc_t pr = make_rsrc(a.part + ((bq0 + hd) * a.n_chunk_max + chunk) * stride, (uint64_t)stride * 4);
        stf(pr, 0, m[i]);
        stf(pr, 4, s[i]);
      }
    }
  }
  const int kg = lane / S::LPR, col0 = 8 * (lane % S::LPR);
  if (kg == 0) {
#pragma unroll
    for (int g = 0; g < GM; ++g) {
      if (g < G) {
        const rsrc_t pr = make_rsrc(a.part + ((bq0 + g) * a.n_chunk_max + chunk) * stride, (uint64_t)stride * 4);
#pragma unroll
        for (int e = 0; e < 8; ++e) stf(pr, (uint32_t)(8 + (col0 + e) * 4), o[g][e]);
      }
    }
  }
}

// One workgroup per (sequence, query head). Thread = (chunk group, column):
// groups stride over the chunk partials with independent loads, then merge
// in group order through LDS.
template <int D>
__global__ __launch_bounds__(kBlock) void decode_combine_kernel(DecodeArgs a) {
  constexpr int NG = kBlock / D;  // chunk groups
  __shared__ float red_m[kBlock / 64];
  __shared__ float red_o[NG][D];
  __shared__ float red_s[NG];
  const int bq = blockIdx.x;
  const int b = bq / a.Hq, qh = bq % a.Hq, h = qh / a.G;
  const int seg = b * a.Hkv + h;
  int64_t r0, r1;
  clamp_segment(a, seg, r0, r1);
  const int64_t len = r1 - r0;
  int64_t nch = (len + a.chunk - 1) / a.chunk;
  if (nch > a.n_chunk_max) nch = a.n_chunk_max;
  const int tid = threadIdx.x, col = tid % D, grp = tid / D;
  const int stride = D + 2;
  const rsrc_t pr = make_rsrc(a.part + (int64_t)bq * a.n_chunk_max * stride, (uint64_t)a.n_chunk_max * stride * 4);
  // global max over the chunks
  float M = -INFINITY;
  for (int64_t c = tid; c < nch; c += kBlock) M = fmaxf(M, ldf(pr, (uint32_t)(c * stride * 4)));
  M = wave_max(M);
  if ((tid & 63) == 0) red_m[tid >> 6] = M;
  __syncthreads();
  M = red_m[0];
#pragma unroll
  for (int u = 1; u < kBlock / 64; ++u) M = fmaxf(M, red_m[u]);
  float S = 0.f, O = 0.f;
  if (M != -INFINITY) {
    int64_t c = grp;
    for (; c + 3 * NG < nch; c += 4 * NG) {
      float mc[4], sc[4], oc[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint32_t base = (uint32_t)((c + u * NG) * stride * 4);
        mc[u] = ldf(pr, base);
        sc[u] = ldf(pr, base + 4);
        oc[u] = ldf(pr, base + 8 + col * 4);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float e = (mc[u] == -INFINITY) ? 0.f : fast_exp2(mc[u] - M);
        S += sc[u] * e;
        O += oc[u] * e;
      }
    }
    for (; c < nch; c += NG) {
      const uint32_t base = (uint32_t)(c * stride * 4);
      const float mc = ldf(pr, base);
      const float e = (mc == -INFINITY) ? 0.f : fast_exp2(mc - M);
      S += ldf(pr, base + 4) * e;
      O += ldf(pr, base + 8 + col * 4) * e;
    }
  }
  red_o[grp][col] = O;
  if (col == 0) red_s[grp] = S;
  __syncthreads();
  if (grp != 0) return;
  S = red_s[0];
  O = red_o[0][col];
#pragma unroll
  for (int g = 1; g < NG; ++g) {
    S += red_s[g];
    O += red_o[g][col];
  }
  const bool empty = !(S > 0.f);
  const float res = empty ? 0.f : O / S;
  if (a.out_dtype == 1) {
    const rsrc_t orr = make_rsrc(static_cast<char*>(a.out) + (int64_t)bq * D * 2, (uint64_t)D * 2);
    const float other = __shfl_xor(res, 1, 64);  // two columns per 32-bit store
    if ((col & 1) == 0) st32(orr, (uint32_t)col * 2, f32_to_bf16_bits(res) | (f32_to_bf16_bits(other) << 16));
  } else {
    const rsrc_t orr = make_rsrc(static_cast<char*>(a.out) + (int64_t)bq * D * 4, (uint64_t)D * 4);
    stf(orr, (uint32_t)col * 4, res);
  }
  if (a.lse_out != nullptr && col == 0) {
    const rsrc_t lr = make_rsrc(a.lse_out, (uint64_t)a.B * a.Hq * 4);
    const float lse = empty ? -INFINITY : (M + fast_log2(S)) * 0.69314718055994530942f;
    stf(lr, (uint32_t)bq * 4, lse);
  }
}

#ifndef SGDKV_DECODE_PF
#define SGDKV_DECODE_PF 2
#endif

// Two steps in flight where the registers allow it (bf16, groups up to 8), else one.
template <typename T, int D>
static void launch_decode_t(const DecodeArgs& a, hipStream_t st) {
  const dim3 grid((a.n_chunk_max + kWaves - 1) / kWaves, a.B * a.Hkv);
  constexpr int PF = sizeof(T) == 2 ? SGDKV_DECODE_PF : 1;
  if (a.G <= 8)
    SGDKV_LAUNCH("decode_split", (decode_split_kernel<T, D, 8, PF>), grid, dim3(kBlock), st, a);
  else
    SGDKV_LAUNCH("decode_split", (decode_split_kernel<T, D, 16, 1>), grid, dim3(kBlock), st, a);
}

hipError_t launch_decode(const DecodeArgs& a, hipStream_t st) {
  if (a.n_chunk_max > 0) {
    if (a.kv_dtype == 1) {
      if (a.D == 128) launch_decode_t<__bf16, 128>(a, st);
      else launch_decode_t<__bf16, 64>(a, st);
    } else {
      if (a.D == 128) launch_decode_t<float, 128>(a, st);
      else launch_decode_t<float, 64>(a, st);
    }
  }
  if (a.D == 128)
    SGDKV_LAUNCH("decode_combine", decode_combine_kernel<128>, dim3(a.B * a.Hq), dim3(kBlock), st, a);
  else
    SGDKV_LAUNCH("decode_combine", decode_combine_kernel<64>, dim3(a.B * a.Hq), dim3(kBlock), st, a);
  return hipGetLastError();
}

}  // namespace sgdkv
