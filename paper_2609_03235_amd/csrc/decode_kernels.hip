// Decode attention over the ragged compressed KV cache (gfx950).
//
// SGD-KV keeps its compressed cache per KV head, before the heads are repeated
// for GQA (Appendix A.2), so one segment of rows serves the G query heads of
// its group. Decode reads each segment once for all G heads:
//
//   decode_split: each wave owns one split of a segment's rows: the splits of
//     a segment take its 16-row steps in turn, so together they sweep the
//     segment front to back. Logits of the G heads against 16 keys at a time
//     are one 16x16 MFMA (the G query rows padded to 16 form the A operand).
//     The wave keeps an online softmax (running max m and sum s per head,
//     base-2 units) and accumulates P.V in fp32 on the vector ALU (bf16 V
//     rows are widened exactly); the next step's K and V are already in
//     flight. The four waves of a workgroup are four neighbouring splits of
//     one segment: at the end they merge their partials through LDS, in wave
//     order, and the workgroup writes one partial (m, s, o[d]) per head.
//   decode_combine: per (sequence, query head), a fixed-order log-sum-exp
//     merge of the workgroup partials; out = o/s, lse = (m + log2 s) * ln 2.
//
// Work is a flattened (chunk, segment) grid, so unequal budgets (one head
// with most of the rows, others with few) still spread over the whole chip.
// Rows appended to a segment after compression (generation) live in a
// separate region per (sequence, KV head) and get splits of their own after
// the compressed ones; the combine merges both.
#include "device_common.h"
#include "mfma_frag.h"
#include "sgdkv_internal.h"

namespace sgdkv {

namespace {
constexpr int kWaves = kDecodeWaves;

// The segment bounds are the same for every lane: taking them from lane 0 lets the
// compiler keep them, and every buffer descriptor built from them, in scalar
// registers (a descriptor in vector registers costs a waterfall loop per load).
__device__ __forceinline__ int64_t uniform64(int64_t v) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)v >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// A decode workgroup's segment and its index in the segment's workgroup layout (x < n_cwg: its
// compressed rows; n_cwg + j: its appended rows), and how many workgroups were launched for the
// segment's compressed rows (ncw): from the compact table, or the (x, segment) grid.
__device__ __forceinline__ void decode_workgroup(const DecodeArgs& a, int& seg, int& x, int& ncw) {
  if (a.compact) {
    const int flat = blockIdx.x;
    int lo = 0, hi = a.B * a.Hkv;  // the last segment lo with wg_start[lo] <= flat (uniform)
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (a.wg_start[mid] <= flat) lo = mid;
      else hi = mid;
    }
    seg = lo;
    ncw = a.wg_start[seg + 1] - a.wg_start[seg] - a.n_new_wg;
    const int local = flat - a.wg_start[seg];
    x = local < ncw ? local : a.n_cwg + (local - ncw);
  } else {
    seg = blockIdx.y;
    x = blockIdx.x;
    ncw = a.n_cwg;
  }
}

// A segment's partial slots: the first one and how many (its launched workgroups, compressed
// rows' first, appended rows' after them).
__device__ __forceinline__ void segment_slots(const DecodeArgs& a, int seg, int64_t& base, int& n) {
  if (a.compact) {
    base = a.wg_start[seg];
    n = a.wg_start[seg + 1] - a.wg_start[seg];
  } else {
    n = a.n_cwg + a.n_new_wg;
    base = (int64_t)seg * n;
  }
}

__device__ __forceinline__ void clamp_segment(const DecodeArgs& a, int seg, int64_t& r0, int64_t& r1) {
  const int nseg = a.B * a.Hkv;
  const rsrc_t orr = make_rsrc(a.offsets, (uint64_t)(nseg + 1) * 8);
  r0 = uniform64((int64_t)ld64(orr, (uint32_t)seg * 8));
  r1 = uniform64((int64_t)ld64(orr, (uint32_t)(seg + 1) * 8));
  r0 = r0 < 0 ? 0 : (r0 > a.total_rows ? a.total_rows : r0);
  r1 = r1 < r0 ? r0 : (r1 > a.total_rows ? a.total_rows : r1);
}
}  // namespace

// Loads of one 16-key step: the K fragments of the MFMA (key lr, k = 32c + 8*lg)
// and this lane's V rows (keys kg + KG*u, columns col0 .. col0+CPL-1). A decode reads each cached
// row once, so the loads carry the non-temporal hint: at 128K x B 8, 256K x B 16 and 1M x B 32
// the split kernel streams 5-6 % faster with it.
template <typename T, int D, int CPL>
struct DecodeStep {
  static constexpr int EB = sizeof(T);
  static constexpr int RB = D * EB;
  static constexpr int NC = D / 32;
  static constexpr int LPR = D / CPL;      // lanes sharing one value row
  static constexpr int KG = 64 / LPR;      // key groups per wave
  static constexpr int VPL = 16 / KG;      // value rows per lane per step
  static constexpr int NW = CPL * EB / 4;  // 32-bit words per lane per value row
  static_assert(NW == 2 || NW % 4 == 0, "value piece");
  Frag<T> kb[NC];
  uint32_t vv[VPL][NW];
  __device__ __forceinline__ void load(const rsrc_t& kr, const rsrc_t& vr, int64_t k0, int lr, int lgp, int kg,
                                       int col0) {
#pragma unroll
    for (int c = 0; c < NC; ++c) kb[c] = gload_frag_nt<T>(kr, (uint32_t)((k0 + lr) * RB + (32 * c + 8 * lgp) * EB));
#pragma unroll
    for (int u = 0; u < VPL; ++u) {
      const uint32_t off = (uint32_t)((k0 + kg + KG * u) * RB + col0 * EB);
      if constexpr (NW == 2) {
        const uint64_t x = ld64_nt(vr, off);
        vv[u][0] = (uint32_t)x;
        vv[u][1] = (uint32_t)(x >> 32);
      } else {
#pragma unroll
        for (int x = 0; x < NW / 4; ++x) {
          const u32x4 y = ld128_nt(vr, off + 16 * x);
          vv[u][4 * x] = y.x;
          vv[u][4 * x + 1] = y.y;
          vv[u][4 * x + 2] = y.z;
          vv[u][4 * x + 3] = y.w;
        }
      }
    }
  }
  __device__ __forceinline__ void value_row(int u, float (&v)[CPL]) const {
    if constexpr (EB == 2) {
#pragma unroll
      for (int x = 0; x < NW; ++x) {
        v[2 * x] = bf16_lo(vv[u][x]);
        v[2 * x + 1] = bf16_hi(vv[u][x]);
      }
    } else {
#pragma unroll
      for (int x = 0; x < NW; ++x) v[x] = __uint_as_float(vv[u][x]);
    }
  }
};

__device__ __forceinline__ void wave_sync() {
  // order this wave's LDS writes before its following LDS reads (other lanes read them)
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
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
template <typename T, int D, int CPL, int GM, int PF, bool EXACT>
__device__ __forceinline__ void decode_chunk(const DecodeArgs& a, float (*pls)[16][16], float (*als)[16],
                                             const rsrc_t& kr, const rsrc_t& vr, int64_t c0, int64_t stride,
                                             int64_t c1, int nsteps,
                                             const Frag<T> (&qa)[D / 32], int lane, float (&m)[4], float (&s)[4],
                                             float (&o)[GM][CPL]) {
  using S = DecodeStep<T, D, CPL>;
  constexpr int NBUF = PF + 1;
  const int lr = lane & 15, lgp = lane >> 4;
  const int kg = lane / S::LPR, col0 = CPL * (lane % S::LPR);
  const float c2 = a.c2;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    m[i] = -INFINITY;
    s[i] = 0.f;
  }
#pragma unroll
  for (int g = 0; g < GM; ++g)
#pragma unroll
    for (int e = 0; e < CPL; ++e) o[g][e] = 0.f;
  // Loads are issued unconditionally (past the last step they repeat it, which the caches
  // serve): a load under a branch makes the compiler wait for every load in flight,
  // prefetches included, before the next use of loaded data.
  const int64_t k_last = c0 + (int64_t)(nsteps - 1) * stride;
  auto step_key = [&](int64_t k) { return k < k_last ? k : k_last; };
  S buf[NBUF];
#pragma unroll
  for (int p = 0; p < PF; ++p) buf[p].load(kr, vr, step_key(c0 + p * stride), lr, lgp, kg, col0);
  for (int it0 = 0; it0 < nsteps; it0 += NBUF) {
#pragma unroll
    for (int u = 0; u < NBUF; ++u) {
      const int it = it0 + u;
      if (it >= nsteps) break;
      const int64_t k0 = c0 + (int64_t)it * stride;
      buf[(u + PF) % NBUF].load(kr, vr, step_key(k0 + PF * stride), lr, lgp, kg, col0);
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
        for (int g = 0; g < GM; ++g) {
          const float al = als[it & 1][g];
#pragma unroll
          for (int e = 0; e < CPL; ++e) o[g][e] *= al;
        }
      }
      // P.V for this lane's value rows and columns
#pragma unroll
      for (int u2 = 0; u2 < S::VPL; ++u2) {
        const int kk = kg + S::KG * u2;
        float v[CPL];
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
        // every row of the padded group: rows past G (zero queries) are never written out,
        // and a branch per head would split the step into blocks that each wait on LDS
#pragma unroll
        for (int g = 0; g < GM; ++g)
#pragma unroll
          for (int e = 0; e < CPL; ++e) o[g][e] = fmaf(pk[g], v[e], o[g][e]);
      }
    }
  }
}

// CPL = value columns per lane; GM = compile-time bound on the group size (8
// or 16); PF = steps of K/V in flight ahead of the one being computed; OCC =
// waves per SIMD the registers are sized for (launch bounds: at least OCC
// waves per execution unit). Each wave owns one split of a segment: split
// index = kWaves*x + wave within the workgroup's region (the
// segment's compressed rows for x < n_cwg, its appended rows after them).
template <typename T, int D, int CPL, int GM, int PF, int OCC>
__global__ __launch_bounds__(kDecodeBlock, OCC) void decode_split_kernel(DecodeArgs a) {
  using S = DecodeStep<T, D, CPL>;
  __shared__ __attribute__((aligned(16))) float pls[kWaves][2][16][16];  // probabilities [key][head]
  __shared__ __attribute__((aligned(16))) float als[kWaves][2][16];      // per-head rescale (exact pass)
  __shared__ float mws[kWaves][16], sws[kWaves][16];                     // each wave's (m, s) per head
  __shared__ __attribute__((aligned(16))) float ows[kWaves][GM][D];      // each wave's o per head

  int seg, x, ncw;
  decode_workgroup(a, seg, x, ncw);
  const int b = seg / a.Hkv, h = seg % a.Hkv;
  const int tid = threadIdx.x, wid = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  int64_t r0, r1;
  clamp_segment(a, seg, r0, r1);
  const int64_t len = r1 - r0;
  // workgroups 0 .. n_cwg-1 cover the segment's compressed rows, the next ones the rows appended
  // since compression. Compact grid: every launched workgroup writes its slot (an empty partial
  // if it has no rows). (x, segment) grid: a workgroup whose first split is empty leaves (uniform
  // over the workgroup). A wave whose own split is empty joins the merge with an empty partial.
  const bool appended = x >= a.n_cwg;
  const int64_t wg = appended ? (int64_t)x - a.n_cwg : (int64_t)x;
  const int64_t chunk = wg * kWaves + wid;  // split index within the region
  const int64_t rows = appended ? a.n_new : len;
  // The compressed rows of a segment are dealt to its nck splits 16 rows at a time (split w
  // takes steps w, w + nck, ...), so the splits of a segment sweep it together from front to
  // back; appended rows form contiguous splits.
  int64_t c0 = 0, stride = 16, c1 = 0;
  int nsteps = 0;
  bool active;
  if (appended) {
    if (!a.compact && wg * kWaves * a.chunk >= rows) return;
    c0 = chunk * a.chunk;
    active = c0 < rows;
    c1 = c0 + a.chunk < rows ? c0 + a.chunk : rows;
    nsteps = active ? (int)((c1 - c0 + 15) / 16) : 0;
  } else {
    // compact grid: four splits per launched workgroup (at most one per step); (x, segment) grid:
    // splits of about a.chunk rows, and device offsets beyond the host's give fewer, longer
    // splits (as many as were launched)
    const int64_t total_steps = (rows + 15) / 16;
    int64_t nck = a.compact ? (int64_t)ncw * kWaves : (rows + a.chunk - 1) / a.chunk;
    if (a.compact) {
      if (nck > total_steps) nck = total_steps;
    } else {
      if (nck > a.n_chunk_max) nck = a.n_chunk_max;
      if (nck > (int64_t)ncw * kWaves) nck = (int64_t)ncw * kWaves;
      if (wg * kWaves >= nck) return;
    }
    active = chunk < nck;
    c0 = chunk * 16;
    stride = nck * 16;
    c1 = rows;
    nsteps = active ? (int)((total_steps - chunk + nck - 1) / nck) : 0;
  }

  const int lr = lane & 15, lgp = lane >> 4;
  const int G = a.G;
  const char* kbase = appended ? static_cast<const char*>(a.k_new) + (int64_t)seg * a.cap * S::RB
                               : static_cast<const char*>(a.k_c) + r0 * S::RB;
  const char* vbase = appended ? static_cast<const char*>(a.v_new) + (int64_t)seg * a.cap * S::RB
                               : static_cast<const char*>(a.v_c) + r0 * S::RB;
  const rsrc_t kr = make_rsrc(kbase, (uint64_t)rows * S::RB);
  const rsrc_t vr = make_rsrc(vbase, (uint64_t)rows * S::RB);
  const rsrc_t qr = make_rsrc(static_cast<const char*>(a.q) + ((int64_t)b * a.Hq + (int64_t)h * G) * S::RB,
                              (uint64_t)G * S::RB);
  Frag<T> qa[S::NC];  // row lr = head; rows >= G read as zeros
#pragma unroll
  for (int c = 0; c < S::NC; ++c) qa[c] = gload_frag<T>(qr, (uint32_t)(lr * S::RB + (32 * c + 8 * lgp) * S::EB));

  float m[4], s[4], o[GM][CPL];
  if (active) {
    decode_chunk<T, D, CPL, GM, PF, false>(a, pls[wid], als[wid], kr, vr, c0, stride, c1, nsteps, qa, lane, m, s, o);
    // 2^64 bounds every probability, so s and o stay finite unless V is huge or the
    // first step's maximum sat far below a later logit: then redo with rescaling
    bool bad = false;
#pragma unroll
    for (int i = 0; i < 4; ++i) bad |= !(s[i] <= 1.8446744073709552e19f);
#pragma unroll
    for (int g = 0; g < GM; ++g)
#pragma unroll
      for (int e = 0; e < CPL; ++e) bad |= !(fabsf(o[g][e]) < INFINITY);
    if (__any(bad))
      decode_chunk<T, D, CPL, GM, PF, true>(a, pls[wid], als[wid], kr, vr, c0, stride, c1, nsteps, qa, lane, m, s, o);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      m[i] = -INFINITY;
      s[i] = 0.f;
    }
#pragma unroll
    for (int g = 0; g < GM; ++g)
#pragma unroll
      for (int e = 0; e < CPL; ++e) o[g][e] = 0.f;
  }

  // Reduce within the wave: the 16 lanes of each head's sum, the KG key groups of o.
#pragma unroll
  for (int i = 0; i < 4; ++i) s[i] = row16_sum(s[i]);
#pragma unroll
  for (int g = 0; g < GM; ++g)
#pragma unroll
    for (int e = 0; e < CPL; ++e) {
      float x = o[g][e];
#pragma unroll
      for (int sft = S::LPR; sft < 64; sft <<= 1) x += __shfl_xor(x, sft, 64);
      o[g][e] = x;
    }
  // Merge the workgroup's splits: each wave leaves its (m, s) and o per head in LDS; then the
  // workgroup's threads merge them in wave order and write one partial per head in the
  // workgroup's slot: (m, s) and o[D] in two arrays, one descriptor each over the segment's slots
  // (per-lane descriptors would cost waterfall loops).
  if (lr == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      mws[wid][4 * lgp + i] = m[i];
      sws[wid][4 * lgp + i] = s[i];
    }
  }
  const int kg = lane / S::LPR, col0 = CPL * (lane % S::LPR);
  if (kg == 0) {
#pragma unroll
    for (int g = 0; g < GM; ++g)
#pragma unroll
      for (int e = 0; e < CPL; e += 4)
        *reinterpret_cast<f32x4*>(&ows[wid][g][col0 + e]) = f32x4{o[g][e], o[g][e + 1], o[g][e + 2], o[g][e + 3]};
  }
  __syncthreads();
  int64_t sbase;
  int nsl;
  segment_slots(a, seg, sbase, nsl);
  const int64_t slot = a.compact ? (int64_t)blockIdx.x - sbase : x;  // within the segment's slots
  const rsrc_t mr = make_rsrc(a.part_ms + sbase * G * 2, (uint64_t)nsl * G * 8);
  const rsrc_t orr = make_rsrc(a.part + sbase * G * D, (uint64_t)nsl * G * D * 4);
  for (int idx = tid; idx < G * D; idx += kDecodeBlock) {
    const int g = idx / D, col = idx % D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, mws[w][g]);
    float O = 0.f, Ssum = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float mw = mws[w][g];
      const float e = mw == -INFINITY ? 0.f : fast_exp2(mw - M);
      O += ows[w][g][col] * e;
      Ssum += sws[w][g] * e;
    }
    stf(orr, (uint32_t)(((slot * G + g) * D + col) * 4), O);
    if (col == 0)
      st64(mr, (uint32_t)((slot * G + g) * 8),
           (uint64_t)__float_as_uint(M) | ((uint64_t)__float_as_uint(Ssum) << 32));
  }
}

// One 256-thread workgroup per (sequence, query head), one pass over the slots: thread (group,
// c4) loads the slots group, group + NG, ... (eight at a time, all in flight together) for
// columns 4*c4 .. 4*c4+3 and merges them with a running reference (the maximum m seen, with the
// sums rescaled when it moves); then the NG group results are merged in group order.
template <int D>
__global__ __launch_bounds__(256) void decode_combine_kernel(DecodeArgs a) {
  constexpr int NT = 256, TPR = D / 4, NG = NT / TPR, U = 8;
  __shared__ float red_m[NG], red_s[NG];
  __shared__ __attribute__((aligned(16))) float red_o[NG][D];
  const int bq = blockIdx.x;
  const int b = bq / a.Hq, qh = bq % a.Hq, h = qh / a.G, g = qh % a.G;
  const int seg = b * a.Hkv + h;
  int64_t sbase;
  int nsl;
  segment_slots(a, seg, sbase, nsl);
  const int64_t ncm = nsl;  // the segment's slots; slot ncm (past the descriptor) reads as zeros
  const int ncw = nsl - a.n_new_wg;  // launched workgroups of the compressed rows
  const int G = a.G;
  const int tid = threadIdx.x, c4 = tid % TPR, grp = tid / TPR;
  const rsrc_t mr = make_rsrc(a.part_ms + sbase * G * 2, (uint64_t)nsl * G * 8);
  const rsrc_t orr = make_rsrc(a.part + sbase * G * D, (uint64_t)nsl * G * D * 4);
  // The first batch of slots is loaded before the segment's length is known, as if every
  // compressed slot were valid, so that its loads travel together with the offsets' instead of
  // after them; slots that turn out invalid are not used.
  uint64_t ms[U];
  u32x4 ov[U];
  auto load_batch = [&](int64_t c, auto&& slot_of) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t sl = slot_of(c + u * NG);
      ms[u] = ld64(mr, (uint32_t)((sl * G + g) * 8));
      ov[u] = ld128(orr, (uint32_t)(((sl * G + g) * D + 4 * c4) * 4));
    }
  };
  load_batch(grp, [&](int64_t c) { return c < ncm ? c : ncm; });
  // Valid slots. Compact grid: all of the segment's (every launched workgroup writes its slot).
  // (x, segment) grid: the workgroups of the segment's nsp splits, then those of its appended
  // splits from slot ncw on; dense index c maps to slot c (c < ncs) or ncw + c - ncs (past nch:
  // the slot past the descriptor, which reads as zeros).
  int64_t ncs = ncm, nch = ncm;
  if (!a.compact) {
    int64_t r0, r1;
    clamp_segment(a, seg, r0, r1);
    const int64_t len = r1 - r0;
    int64_t nsp = (len + a.chunk - 1) / a.chunk;
    if (nsp > a.n_chunk_max) nsp = a.n_chunk_max;
    if (nsp > (int64_t)ncw * kWaves) nsp = (int64_t)ncw * kWaves;  // as the split kernel clamps
    ncs = (nsp + kWaves - 1) / kWaves;
    nch = ncs + (a.n_new_chunks + kWaves - 1) / kWaves;
    if (a.n_new_chunks > 0) load_batch(grp, [&](int64_t c) { return c >= nch ? ncm : (c < ncs ? c : ncw + (c - ncs)); });
  }
  auto slot = [&](int64_t c) { return c >= nch ? ncm : (c < ncs ? c : ncw + (c - ncs)); };
  float M = -INFINITY, S = 0.f, O[4] = {0.f, 0.f, 0.f, 0.f};
  for (int64_t c = grp; c < nch; c += U * NG) {
    if (c != grp) load_batch(c, slot);
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (!(c + u * NG < nch)) {  // a slot past the segment's (possibly stale memory): m = -inf, s = o = 0
        ms[u] = 0xFF800000ull;
        ov[u] = u32x4{0u, 0u, 0u, 0u};
      }
    float Mn = M;
#pragma unroll
    for (int u = 0; u < U; ++u) Mn = fmaxf(Mn, __uint_as_float((uint32_t)ms[u]));
    if (Mn != -INFINITY) {
      const float r = M == -INFINITY ? 0.f : fast_exp2(M - Mn);
      S *= r;
#pragma unroll
      for (int k = 0; k < 4; ++k) O[k] *= r;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float mc = __uint_as_float((uint32_t)ms[u]), sc = __uint_as_float((uint32_t)(ms[u] >> 32));
        const float e = mc != -INFINITY ? fast_exp2(mc - Mn) : 0.f;
        S += sc * e;
        O[0] += __uint_as_float(ov[u].x) * e;
        O[1] += __uint_as_float(ov[u].y) * e;
        O[2] += __uint_as_float(ov[u].z) * e;
        O[3] += __uint_as_float(ov[u].w) * e;
      }
      M = Mn;
    }
  }
  *reinterpret_cast<f32x4*>(&red_o[grp][4 * c4]) = f32x4{O[0], O[1], O[2], O[3]};
  if (c4 == 0) {
    red_m[grp] = M;
    red_s[grp] = S;
  }
  __syncthreads();
  if (tid >= D) return;
  const int col = tid;
  float Mf = red_m[0];
#pragma unroll
  for (int g = 1; g < NG; ++g) Mf = fmaxf(Mf, red_m[g]);
  float Sf = 0.f, Oc = 0.f;
  if (Mf != -INFINITY) {
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const float e = red_m[g] == -INFINITY ? 0.f : fast_exp2(red_m[g] - Mf);
      Sf += red_s[g] * e;
      Oc += red_o[g][col] * e;
    }
  }
  const bool empty = !(Sf > 0.f);
  const float res = empty ? 0.f : Oc / Sf;
  if (a.out_dtype == 1) {
    const rsrc_t outr = make_rsrc(static_cast<char*>(a.out) + (int64_t)bq * D * 2, (uint64_t)D * 2);
    const float other = __shfl_xor(res, 1, 64);  // two columns per 32-bit store
    if ((col & 1) == 0) st32(outr, (uint32_t)col * 2, f32_to_bf16_bits(res) | (f32_to_bf16_bits(other) << 16));
  } else {
    const rsrc_t outr = make_rsrc(static_cast<char*>(a.out) + (int64_t)bq * D * 4, (uint64_t)D * 4);
    stf(outr, (uint32_t)col * 4, res);
  }
  if (a.lse_out != nullptr && col == 0) {
    const rsrc_t lr = make_rsrc(a.lse_out, (uint64_t)a.B * a.Hq * 4);
    const float lse = empty ? -INFINITY : (Mf + fast_log2(Sf)) * 0.69314718055994530942f;
    stf(lr, (uint32_t)bq * 4, lse);
  }
}

#ifndef SGDKV_DECODE_PF
#define SGDKV_DECODE_PF 1
#endif
#ifndef SGDKV_DECODE_CPL
#define SGDKV_DECODE_CPL 8
#endif
#ifndef SGDKV_DECODE_OCC
#define SGDKV_DECODE_OCC 2
#endif

// One step of K/V in flight ahead of the one being computed (more measured no faster).
template <typename T, int D>
static void launch_decode_t(const DecodeArgs& a, hipStream_t st) {
  const dim3 grid = a.compact ? dim3((unsigned)a.wg_start[a.B * a.Hkv]) : dim3(a.n_cwg + a.n_new_wg, a.B * a.Hkv);
  constexpr bool wide = sizeof(T) == 2;
  constexpr int PF = wide ? SGDKV_DECODE_PF : 1;
  constexpr int CPL = wide ? SGDKV_DECODE_CPL : 8;
  constexpr int OCC = wide ? SGDKV_DECODE_OCC : 2;
  if (a.G <= 8)
    SGDKV_LAUNCH("decode_split", (decode_split_kernel<T, D, CPL, 8, PF, OCC>), grid, dim3(kDecodeBlock), st, a);
  else
    SGDKV_LAUNCH("decode_split", (decode_split_kernel<T, D, 8, 16, 1, 2>), grid, dim3(kDecodeBlock), st, a);
}

// Copies one token's K rows (blockIdx.y = 0) or V rows (1), [B*Hkv][d] each, into row `slot`
// of every (b, h) of the appended regions: one 16-byte vector per thread.
__global__ __launch_bounds__(kBlock) void append_kernel(DecodeArgs a, const void* k_step, const void* v_step,
                                                         void* k_new, void* v_new, int64_t slot) {
  const int rb = a.D * (a.kv_dtype == 1 ? 2 : 4);
  const int v16 = rb / 16;
  const int64_t nseg = (int64_t)a.B * a.Hkv;
  const int64_t r = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (r >= nseg * v16) return;
  const bool is_v = blockIdx.y == 1;
  const int64_t seg = r / v16, c = r % v16;
  const rsrc_t src = make_rsrc(is_v ? v_step : k_step, (uint64_t)nseg * rb);
  const rsrc_t dst = make_rsrc(is_v ? v_new : k_new, (uint64_t)nseg * a.cap * rb);
  st128(dst, (uint32_t)((seg * a.cap + slot) * rb + c * 16), ld128(src, (uint32_t)(seg * rb + c * 16)));
}

hipError_t launch_append(const DecodeArgs& a, const void* k_step, const void* v_step, void* k_new, void* v_new,
                         int64_t slot, hipStream_t st) {
  const int64_t n = (int64_t)a.B * a.Hkv * (a.D * (a.kv_dtype == 1 ? 2 : 4) / 16);
  SGDKV_LAUNCH("append", append_kernel, dim3((unsigned)((n + kBlock - 1) / kBlock), 2), dim3(kBlock), st, a, k_step,
               v_step, k_new, v_new, slot);
  return hipGetLastError();
}

hipError_t launch_decode(const DecodeArgs& a, hipStream_t st) {
  if (a.compact ? a.wg_start[a.B * a.Hkv] > 0 : a.n_chunk_max + a.n_new_chunks > 0) {
    if (a.kv_dtype == 1) {
      if (a.D == 128) launch_decode_t<__bf16, 128>(a, st);
      else launch_decode_t<__bf16, 64>(a, st);
    } else {
      if (a.D == 128) launch_decode_t<float, 128>(a, st);
      else launch_decode_t<float, 64>(a, st);
    }
  }
  if (a.D == 128)
    SGDKV_LAUNCH("decode_combine", decode_combine_kernel<128>, dim3(a.B * a.Hq), dim3(256), st, a);
  else
    SGDKV_LAUNCH("decode_combine", decode_combine_kernel<64>, dim3(a.B * a.Hq), dim3(256), st, a);
  return hipGetLastError();
}

}  // namespace sgdkv
