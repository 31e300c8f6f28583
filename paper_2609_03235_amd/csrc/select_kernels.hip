// Pooling, per-head top-k selection and gather for SGD-KV (gfx950).
//
// For KV head h with budget b_h, SGD-KV keeps the b_sink initial rows, the
// b_window most recent rows (Sec. 3.3) and, in between, the m_h = b_h -
// b_sink - b_window candidates with the largest pooled window score
// (Sec. 3.3, last paragraph). The kept rows are copied, per KV head and
// before GQA repetition (Appendix A.2), into a ragged cache.
//
// Selection is an exact, deterministic top-k with ties to the lower
// position. Scores are non-negative fp32, so their bit patterns order like
// the values. An MSB-first radix select (four 8-bit digits) finds the k-th
// largest pattern tau and how many of the rows equal to tau are kept (q);
// the compaction then keeps every candidate above tau and the first q equal
// to tau in position order. Histograms use integer atomics only; everything
// else is fixed-order, so results are bitwise reproducible.
//
// Kernels (grid y = segment b*Hkv + h):
//   select_init    zero the histograms, write the offsets (when the column-sum pass,
//                  which otherwise does it, does not run)
//   radix_pass<p>  digit-p histogram of candidates matching the digits
//                  before it (each workgroup picks those from the earlier
//                  histograms itself); the last pass also keeps each chunk's
//                  histogram and its count above the prefix; pass 0 also pools:
//                  pooled_j = (1/k_p) sum_{|t-j|<=r} a_t (zero outside), where
//                  a_t combines the column-sum partials of the score pass's
//                  row splits in split order (their sum; their maximum for
//                  the Ipt. max aggregation)
//   compact        picks tau and q from the four histograms, then the ordered
//                  ballot/prefix compaction of a chunk -> kept_pos (the rows kept
//                  before the chunk from the last radix pass's chunk histograms)
//   copy_rows      K and V rows of the kept positions -> the ragged cache
#include <algorithm>

#include "device_common.h"
#include "sgdkv_internal.h"
#include "segment_init.h"

namespace sgdkv {

namespace {

// Radix-select state of a segment: the digits of tau found so far (prefix,
// under mask) and how many rows are still to place among the candidates that
// match them; after the fourth digit, prefix = tau and rem = q.
struct SegState {
  uint32_t prefix, mask, rem;
};

// Adds one to bin `bin` of an LDS histogram for every lane with `valid` (call
// with the whole wave). Scores crowd into a few bins, where one atomic per
// lane would serialise: the wave takes the distinct bins in turn and adds each
// bin's lane count with one atomic; after four bins the remaining lanes add
// one by one.
__device__ __forceinline__ void hist_add(uint32_t* lh, uint32_t bin, bool valid) {
  const int lane = threadIdx.x & 63;
  unsigned long long pending = __ballot(valid);
#pragma unroll
  for (int round = 0; round < 4; ++round) {
    if (pending == 0ull) return;  // uniform
    const int leader = __builtin_ctzll(pending);
    const uint32_t lb = (uint32_t)__shfl((int)bin, leader, 64);
    const unsigned long long same = __ballot(bin == lb) & pending;
    if (lane == leader) atomicAdd(&lh[lb], (uint32_t)__popcll(same));
    pending &= ~same;
  }
  if ((pending >> lane) & 1ull) atomicAdd(&lh[bin], 1u);
}

// Exclusive rank of `flag` among the threads of a 256-thread block, and the
// block total. Uses wave ballots plus one LDS exchange; `wtot` holds 4 words.
__device__ __forceinline__ uint32_t block_rank(bool flag, uint32_t* wtot, uint32_t& total) {
  const int tid = threadIdx.x, wid = tid >> 6, lane = tid & 63;
  const unsigned long long bal = __ballot(flag);
  const uint32_t below = (uint32_t)__popcll(bal & ((1ull << lane) - 1ull));
  if (lane == 0) wtot[wid] = (uint32_t)__popcll(bal);
  __syncthreads();
  uint32_t before = 0, tot = 0;
#pragma unroll
  for (int u = 0; u < kBlock / 64; ++u) {
    const uint32_t t = wtot[u];
    before += (u < wid) ? t : 0u;
    tot += t;
  }
  __syncthreads();
  total = tot;
  return before + below;
}

}  // namespace

// Only when no column-sum pass ran (no scored keys): that pass otherwise does this set-up.
__global__ __launch_bounds__(kBlock) void select_init_kernel(CompressArgs a) { init_segment(a, blockIdx.x); }

// The radix state after digits 0 .. NPASS-1: every digit is picked from its
// histogram (complete once the pass that built it has ended) as the unique
// digit t with S(t) >= rem > S(t+1), S the suffix sums of the bins; rem then
// drops by S(t+1). Runs in every workgroup that needs it (256 threads; `sh`
// holds 256 + 8 words of LDS); the result is the same in all of them.
template <int NPASS>
__device__ __forceinline__ SegState derive_state(const CompressArgs& a, int seg, uint32_t* sh) {
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  SegState st;
  st.prefix = 0u;
  st.mask = 0u;
  st.rem = (uint32_t)a.m[seg % a.Hkv];
  if (NPASS == 0 || st.rem == 0) return st;
  const rsrc_t hr = make_rsrc(a.hist + (int64_t)seg * 4 * 256, 4 * 256 * 4);
  uint32_t hv[NPASS > 0 ? NPASS : 1];
#pragma unroll
  for (int p = 0; p < NPASS; ++p) hv[p] = ld32(hr, (p * 256 + tid) * 4);  // all issued before any use
#pragma unroll
  for (int p = 0; p < NPASS; ++p) {
    const int shift = 24 - 8 * p;
    // suffix sums: within the wave (lanes above), then the waves above
    uint32_t v = hv[p];
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t t = __shfl_down(v, o, 64);
      v += lane + o < 64 ? t : 0u;
    }
    if (lane == 0) sh[256 + wid] = v;
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kBlock / 64; ++u) v += u > wid ? sh[256 + u] : 0u;
    const uint32_t S = v, Sn = v - hv[p];
    if (S >= st.rem && Sn < st.rem) {  // exactly one digit satisfies this
      sh[256 + 4] = (uint32_t)tid;
      sh[256 + 5] = Sn;
    }
    __syncthreads();
    const uint32_t dg = sh[256 + 4], below = sh[256 + 5];
    __syncthreads();
    st.prefix |= dg << shift;
    st.mask |= 0xFFu << shift;
    st.rem -= below;
  }
  return st;
}

// Pooling and the histogram of one digit of the radix select. Workgroup
// (x, seg) covers the scored positions [j0, j1) = [x*hist_chunk,
// (x+1)*hist_chunk) of segment seg.
//   POOL (digit 0 only): pooled_j = (1/k_p) sum_{t=-r..r} a_{j+t}, added in
//     order of t, zeros outside [0, n_scored); the column sums of
//     [j0-r, j1+r) are staged in LDS when r <= kPoolHalo.
//   HIST: histogram of digit PASS over the candidates [s, C-W) of the range
//     whose higher digits match the prefix found so far, added to the
//     segment's histogram with integer atomics.
//   KP: the pooling width when it is one of the widths built in (1..15, odd): each thread
//     then pools four consecutive positions from values it reads once with 16-byte LDS
//     loads (same additions in the same order as the general loop); 0: any width.
template <int PASS, bool POOL, bool HIST, int KP = 0>
__global__ __launch_bounds__(kBlock) void radix_pass_kernel(CompressArgs a) {
  __shared__ uint32_t lh[256 + 8];
  __shared__ __attribute__((aligned(16))) float win[POOL ? kHistChunkMax + 2 * kPoolHalo + 16 : 1];
  const int seg = blockIdx.y, tid = threadIdx.x;
  const SegState st = derive_state<PASS>(a, seg, lh);
  const bool hist = HIST && st.rem != 0;  // uniform per segment: nothing (left) to choose otherwise
  if (!POOL && !hist) return;
  constexpr int shift = 24 - 8 * PASS;
  lh[tid] = 0;
  const int64_t j0 = (int64_t)blockIdx.x * a.hist_chunk;
  const int64_t j1 = j0 + a.hist_chunk < a.n_scored ? j0 + a.hist_chunk : a.n_scored;
  const int64_t cbeg = a.s, cend = a.C - a.W;
  const rsrc_t pr = make_rsrc(a.pooled + (int64_t)seg * a.n_scored, (uint64_t)a.n_scored * 4);
  // Loads go out in batches of U per thread, issued before any is used: positions past the
  // range read whatever the descriptor gives (zero past its end) and are not used.
  constexpr int U = 8;
  if constexpr (POOL) {
    const int nseg = a.B * a.Hkv;
    const bool maxg = a.agg == 1;
    auto split_rsrc = [&](int p) {
      return make_rsrc(a.colsum + ((int64_t)p * nseg + seg) * a.n_scored, (uint64_t)a.n_scored * 4);
    };
    const rsrc_t cr = split_rsrc(0);
    // a_t at byte offset off: the partials of all row splits, combined in split order
    auto colsum_at = [&](uint32_t off) {
      float x = ldf(cr, off);
      for (int p = 1; p < a.n_rsplit; ++p) {
        const float y = ldf(split_rsrc(p), off);
        x = maxg ? fmaxf(x, y) : x + y;
      }
      return x;
    };
    const int r = (a.kp - 1) / 2;
    const float fk = (float)a.kp;
    const bool staged = r <= kPoolHalo;
    if (staged) {
      // positions before 0 or past n_scored fall outside the descriptor and read as 0
      const int64_t n = (j1 - j0) + 2 * r;
      for (int64_t i0 = 0; i0 < n; i0 += U * kBlock) {
        float x[U];
#pragma unroll
        for (int u = 0; u < U; ++u) x[u] = ldf(cr, (uint32_t)((j0 - r + i0 + tid + u * kBlock) * 4));
        for (int p = 1; p < a.n_rsplit; ++p) {  // the other row splits' partials, in split order
          const rsrc_t cp = split_rsrc(p);
          float y[U];
#pragma unroll
          for (int u = 0; u < U; ++u) y[u] = ldf(cp, (uint32_t)((j0 - r + i0 + tid + u * kBlock) * 4));
#pragma unroll
          for (int u = 0; u < U; ++u) x[u] = maxg ? fmaxf(x[u], y[u]) : x[u] + y[u];
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
          if (i0 + tid + u * kBlock < n) win[i0 + tid + u * kBlock] = x[u];
      }
    }
    __syncthreads();
    if constexpr (KP > 0) {
      // positions j .. j+3 need win[j - j0 .. j - j0 + 3 + 2R]: NV 16-byte reads from a
      // 16-byte aligned start (the last few values are read past the staged ones and unused)
      constexpr int R = (KP - 1) / 2, NV = (4 + 2 * R + 3) / 4;
      const bool aligned = (((int64_t)seg * a.n_scored) & 3) == 0;  // pooled rows start 16-byte aligned
      for (int64_t jb = j0; jb < j1; jb += 4 * kBlock) {  // uniform trip count
        const int64_t j = jb + 4 * tid;
        float x[4 * NV];
#pragma unroll
        for (int q = 0; q < NV; ++q) {
          const f32x4 w4 = *reinterpret_cast<const f32x4*>(win + (j - j0) + 4 * q);
          x[4 * q] = w4.x;
          x[4 * q + 1] = w4.y;
          x[4 * q + 2] = w4.z;
          x[4 * q + 3] = w4.w;
        }
        float v[4];
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          float sum = 0.f;
#pragma unroll
          for (int t = 0; t <= 2 * R; ++t) sum += x[p + t];
          v[p] = sum / fk;
        }
        if (aligned && j + 3 < j1) {
          u32x4 o;
          o.x = __float_as_uint(v[0]);
          o.y = __float_as_uint(v[1]);
          o.z = __float_as_uint(v[2]);
          o.w = __float_as_uint(v[3]);
          st128(pr, (uint32_t)(j * 4), o);
        } else {
#pragma unroll
          for (int p = 0; p < 4; ++p)
            if (j + p < j1) stf(pr, (uint32_t)((j + p) * 4), v[p]);
        }
        if (hist) {
#pragma unroll
          for (int p = 0; p < 4; ++p) {
            const uint32_t bits = __float_as_uint(v[p]);
            const int64_t jp = j + p;
            hist_add(lh, (bits >> shift) & 255u,
                     jp < j1 && jp >= cbeg && jp < cend && (bits & st.mask) == st.prefix);
          }
        }
      }
    } else {
      for (int64_t jb = j0; jb < j1; jb += kBlock) {  // uniform trip count: hist_add needs the whole wave
        const int64_t j = jb + tid;
        const bool in = j < j1;
        float v = 0.f;
        if (in) {
          float sum = 0.f;
          if (staged) {
            const float* wp = win + (j - j0);
            for (int t = 0; t <= 2 * r; ++t) sum += wp[t];
          } else {
            for (int t = -r; t <= r; ++t) sum += colsum_at((uint32_t)((j + t) * 4));
          }
          v = sum / fk;
          stf(pr, (uint32_t)(j * 4), v);
        }
        if (hist) {
          const uint32_t bits = __float_as_uint(v);
          hist_add(lh, (bits >> shift) & 255u, in && j >= cbeg && j < cend && (bits & st.mask) == st.prefix);
        }
      }
    }
  } else {
    __syncthreads();
    const int64_t c0 = j0 > cbeg ? j0 : cbeg, c1 = j1 < cend ? j1 : cend;
    uint32_t above = 0;  // the last pass: candidates above the 24-bit prefix (all of them above tau)
    for (int64_t jb = c0; jb < c1; jb += U * kBlock) {
      uint32_t x[U];
#pragma unroll
      for (int u = 0; u < U; ++u) x[u] = ld32(pr, (uint32_t)((jb + tid + u * kBlock) * 4));
      // few candidates still match the prefix here, spread over more bins: one atomic per lane
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const bool in = jb + tid + u * kBlock < c1;
        if (in && (x[u] & st.mask) == st.prefix) atomicAdd(&lh[(x[u] >> shift) & 255u], 1u);
        if (PASS == 3) above += in && (x[u] & st.mask) > st.prefix;
      }
    }
    if constexpr (PASS == 3) {
      // the chunk's histogram and its count above, for the compaction's running totals
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) above += __shfl_xor(above, o, 64);
      if ((tid & 63) == 0) lh[256 + (tid >> 6)] = above;
      __syncthreads();
      const rsrc_t chr = make_rsrc(a.chunk_hist + ((int64_t)seg * a.n_hist_chunks + blockIdx.x) * kChunkHistWords,
                                   kChunkHistWords * 4);
      st32(chr, (uint32_t)tid * 4u, lh[tid]);
      if (tid == 0) st32(chr, 256u * 4u, lh[256] + lh[257] + lh[258] + lh[259]);
    }
  }
  if (!hist) return;
  __syncthreads();
  const uint32_t v = lh[tid];
  if (v) atomicAdd(a.hist + ((int64_t)seg * 4 + PASS) * 256 + tid, v);
}

// Ordered compaction of one chunk of positions (the chunks of the radix passes, then chunks of
// window rows): writes the prompt positions of the kept rows (ascending) into the segment's
// slice of kept_pos. tau and q come from the segment's four digit histograms; the rows the
// chunks before this one keep, from their positions (sink and window rows) and, for their
// candidates, the last pass's chunk histograms: those above tau's top 24 bits, those matching
// them with a last digit above tau's, and those equal to tau (of which the first q are kept).
__global__ __launch_bounds__(kBlock) void compact_kernel(CompressArgs a) {
  __shared__ uint32_t wt0[kBlock / 64], wt1[kBlock / 64];
  __shared__ uint32_t pre[3][kBlock / 64];
  __shared__ uint32_t sh[256 + 8];
  const int seg = blockIdx.y, b = seg / a.Hkv, h = seg % a.Hkv;
  const int chunk = blockIdx.x;
  const int tid = threadIdx.x;
  const SegState st = derive_state<4>(a, seg, sh);
  const bool active = a.m[h] > 0;
  const uint32_t tau = st.prefix;
  const uint32_t q = active ? st.rem : 0u;
  const int64_t j0 = (int64_t)chunk * a.hist_chunk;
  const int64_t j1 = j0 + a.hist_chunk < a.C ? j0 + a.hist_chunk : a.C;
  const int64_t cend = a.C - a.W;

  // totals of the chunks before this one: sink/window rows, > tau, == tau
  const uint32_t F = (uint32_t)((j0 < a.s ? j0 : a.s) + (j0 > cend ? j0 - cend : 0));
  uint32_t g = 0, e = 0;
  if (active) {
    const int nc = chunk < a.n_hist_chunks ? chunk : a.n_hist_chunks;
    const rsrc_t chr = make_rsrc(a.chunk_hist + (int64_t)seg * a.n_hist_chunks * kChunkHistWords,
                                 (uint64_t)a.n_hist_chunks * kChunkHistWords * 4);
    const uint32_t dt = tau & 255u;
    constexpr int U = 32;  // loads in flight per thread
    uint32_t bin = 0, above = 0;
    for (int c0 = 0; c0 < nc; c0 += U) {
      uint32_t x[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c = c0 + u < nc ? c0 + u : nc;  // past the chunks before this one: read, not used
        x[u] = ld32(chr, (uint32_t)(c * kChunkHistWords + tid) * 4u);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) bin += c0 + u < nc ? x[u] : 0u;
    }
    for (int c = tid; c < nc; c += kBlock) above += ld32(chr, (uint32_t)(c * kChunkHistWords + 256) * 4u);
    g = above + (tid > (int)dt ? bin : 0u);
    e = tid == (int)dt ? bin : 0u;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    g += __shfl_xor(g, o, 64);
    e += __shfl_xor(e, o, 64);
  }
  if ((tid & 63) == 0) {
    pre[1][tid >> 6] = g;
    pre[2][tid >> 6] = e;
  }
  __syncthreads();
  uint32_t Gt = 0, E = 0;
#pragma unroll
  for (int u = 0; u < kBlock / 64; ++u) {
    Gt += pre[1][u];
    E += pre[2][u];
  }
  uint32_t run_keep = F + Gt + (E < q ? E : q);
  uint32_t run_eq = E;

  const int64_t seg_off = (int64_t)b * a.T_layer + a.prefix[h];
  const int64_t seg_len = a.prefix[h + 1] - a.prefix[h];
  const rsrc_t kp = make_rsrc(a.kept_pos + seg_off, (uint64_t)seg_len * 4);
  const rsrc_t pr = make_rsrc(a.pooled + (int64_t)seg * a.n_scored, (uint64_t)a.n_scored * 4);

  // positions in order, 256 at a time; the scores of the next U*256 are loaded together first
  constexpr int U = 8;
  for (int64_t ubase = j0; ubase < j1; ubase += U * kBlock) {
    uint32_t x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) x[u] = ld32(pr, (uint32_t)((ubase + u * kBlock + tid) * 4));
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t base = ubase + u * kBlock;
    if (base >= j1) break;  // uniform
    const int64_t j = base + tid;
    const bool inr = j < j1;
    const bool fixed = inr && (j < a.s || j >= cend);
    const bool cand = inr && !fixed && active;
    const uint32_t bits = cand ? x[u] : 0u;
    const bool gt = cand && bits > tau;
    const bool eq = cand && bits == tau;
    uint32_t n_eq, n_keep;
    const uint32_t eq_rank = run_eq + block_rank(eq, wt0, n_eq);
    const bool keep = fixed || gt || (eq && eq_rank < q);
    const uint32_t r = block_rank(keep, wt1, n_keep);
    if (keep) st32(kp, (run_keep + r) * 4u, (uint32_t)j);
    run_eq += n_eq;
    run_keep += n_keep;
  }
  }
}

// Copies the kept K and V rows into the ragged cache. A work item is
// kCopyRows output rows of one segment (item = seg * copy_blocks + block);
// workgroups take items in a grid-stride loop, so the grid may be smaller
// than the item count (the library shrinks it when the copy runs beside
// other work). Every thread keeps several 16-byte loads in flight before
// storing. RB = bytes per row. Loads and stores carry the non-temporal hint: beside the next
// layer's window scoring, whose second pass re-reads the ends of the first pass's key chunks from
// the last-level cache, the copy then does not push those keys out (the 28-layer 128K x B 8 step
// 1 % faster); and the copied rows do not linger dirty in the caches, where their write-back
// would compete with the decode that reads them next (a 1M x B 32 layer: copy 6.64 -> 6.26 ms,
// decode 2.74 -> 2.60 ms).
template <int RB>
__global__ __launch_bounds__(kBlock) void copy_rows_kernel(CompressArgs a) {
  constexpr int NT = kNonTemporal;  // buffer cache policy
  constexpr int V16 = RB / 16;                        // 16-byte pieces per row
  constexpr int PER = kCopyRows * V16 / kBlock;       // pieces per thread per tensor
  static_assert(PER >= 1 && (kCopyRows * V16) % kBlock == 0, "copy tile must split evenly");
  const int64_t items = (int64_t)a.copy_blocks * a.B * a.Hkv;
  for (int64_t item = blockIdx.x; item < items; item += gridDim.x) {
    const int seg = (int)(item / a.copy_blocks), b = seg / a.Hkv, h = seg % a.Hkv;
    const int64_t seg_len = a.prefix[h + 1] - a.prefix[h];
    const int64_t row0 = (item % a.copy_blocks) * kCopyRows;
    if (row0 >= seg_len) continue;  // uniform per workgroup
    const int64_t seg_off = (int64_t)b * a.T_layer + a.prefix[h];
    const rsrc_t kp = make_rsrc(a.kept_pos + seg_off, (uint64_t)seg_len * 4);
    const rsrc_t ko = make_rsrc(static_cast<char*>(a.k_out) + seg_off * RB, (uint64_t)seg_len * RB);
    const rsrc_t vo = make_rsrc(static_cast<char*>(a.v_out) + seg_off * RB, (uint64_t)seg_len * RB);
    const rsrc_t ki = make_rsrc(static_cast<const char*>(a.k) + (int64_t)seg * a.C * RB, (uint64_t)a.C * RB);
    const rsrc_t vi = make_rsrc(static_cast<const char*>(a.v) + (int64_t)seg * a.C * RB, (uint64_t)a.C * RB);
    u32x4 kx[PER], vx[PER];
    uint32_t dst[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int x = threadIdx.x + u * kBlock;
      const int r = x / V16, c16 = x % V16;
      const int64_t row = row0 + r;  // rows past the segment read position 0 and store out of range
      const uint32_t pos = ld32(kp, (uint32_t)(row * 4));
      const uint32_t src = pos * RB + c16 * 16;
      dst[u] = (uint32_t)(row * RB + c16 * 16);
      kx[u] = __builtin_amdgcn_raw_buffer_load_b128(ki, (int)src, 0, NT);
      vx[u] = __builtin_amdgcn_raw_buffer_load_b128(vi, (int)src, 0, NT);
    }
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      __builtin_amdgcn_raw_buffer_store_b128(kx[u], ko, (int)dst[u], 0, NT);
      __builtin_amdgcn_raw_buffer_store_b128(vx[u], vo, (int)dst[u], 0, NT);
    }
  }
}

// Pooling (+ the digit-0 histogram) with the width built in where one is.
template <bool HIST>
static void launch_pool(const CompressArgs& a, dim3 grid, hipStream_t st) {
  const dim3 blk(kBlock);
  const char* name = HIST ? "pool_radix_hist" : "pool";
  switch (a.kp) {
    case 1: SGDKV_LAUNCH(name, (radix_pass_kernel<0, true, HIST, 1>), grid, blk, st, a); break;
    case 3: SGDKV_LAUNCH(name, (radix_pass_kernel<0, true, HIST, 3>), grid, blk, st, a); break;
    case 5: SGDKV_LAUNCH(name, (radix_pass_kernel<0, true, HIST, 5>), grid, blk, st, a); break;
    case 7: SGDKV_LAUNCH(name, (radix_pass_kernel<0, true, HIST, 7>), grid, blk, st, a); break;
    case 9: SGDKV_LAUNCH(name, (radix_pass_kernel<0, true, HIST, 9>), grid, blk, st, a); break;
    case 11: SGDKV_LAUNCH(name, (radix_pass_kernel<0, true, HIST, 11>), grid, blk, st, a); break;
    case 13: SGDKV_LAUNCH(name, (radix_pass_kernel<0, true, HIST, 13>), grid, blk, st, a); break;
    case 15: SGDKV_LAUNCH(name, (radix_pass_kernel<0, true, HIST, 15>), grid, blk, st, a); break;
    default: SGDKV_LAUNCH(name, (radix_pass_kernel<0, true, HIST, 0>), grid, blk, st, a); break;
  }
}

hipError_t launch_select(const CompressArgs& a, bool scores_only, hipStream_t st) {
  const int nseg = a.B * a.Hkv;
  const dim3 blk(kBlock);
  if (a.n_col_chunks == 0) SGDKV_LAUNCH("select_init", select_init_kernel, dim3(nseg), blk, st, a);
  const dim3 hgrid(a.n_hist_chunks, nseg);
  const bool cands = a.C - a.s - a.W > 0;
  if (scores_only || !cands) {
    if (a.n_hist_chunks > 0) launch_pool<false>(a, hgrid, st);
    if (scores_only) return hipGetLastError();
  } else {
    launch_pool<true>(a, hgrid, st);
    SGDKV_LAUNCH("radix_hist", (radix_pass_kernel<1, false, true>), hgrid, blk, st, a);
    SGDKV_LAUNCH("radix_hist", (radix_pass_kernel<2, false, true>), hgrid, blk, st, a);
    SGDKV_LAUNCH("radix_hist", (radix_pass_kernel<3, false, true>), hgrid, blk, st, a);
  }
  SGDKV_LAUNCH("compact", compact_kernel, dim3(a.n_cmp_chunks, nseg), blk, st, a);
  return hipGetLastError();
}

hipError_t launch_gather(const CompressArgs& a, int max_blocks, hipStream_t st) {
  const int64_t items = (int64_t)a.copy_blocks * a.B * a.Hkv;
  if (items == 0) return hipSuccess;
  // a full grid is capped too (the loop covers the rest), keeping blocks x threads below 2^32
  const unsigned grid = (unsigned)std::min<int64_t>(items, max_blocks > 0 ? max_blocks : (1 << 20));
  const dim3 blk(kBlock);
  switch (a.D * (a.dtype == 1 ? 2 : 4)) {
    case 128: SGDKV_LAUNCH("gather", copy_rows_kernel<128>, dim3(grid), blk, st, a); break;
    case 256: SGDKV_LAUNCH("gather", copy_rows_kernel<256>, dim3(grid), blk, st, a); break;
    case 512: SGDKV_LAUNCH("gather", copy_rows_kernel<512>, dim3(grid), blk, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace sgdkv
