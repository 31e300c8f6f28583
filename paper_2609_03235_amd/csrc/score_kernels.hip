// Observation-window scoring for SGD-KV token selection (gfx950).
//
// Token selection keeps, inside each KV head's budget, the keys with the
// largest cumulative attention of a final observation window (SGD-KV
// Sec. 3.3, last paragraph, SnapKV-style; Sec. 5 Query-Aware window). Window
// row i of query head q sits at prompt position C-w+i and attends causally to
// keys 0..C-w+i. For each KV head the G*w rows of its query group are one
// dense block R x d, so the logits of a key tile are an R x 16 MFMA product.
//
//   pass 1 (lse_kernel + lse_merge_kernel): base-2 log-sum-exp of every
//     window row over its causal keys. Each workgroup covers one chunk of
//     keys and leaves per-row partials (m, s); the merge combines the chunks
//     in a fixed order, in fp64.
//   pass 2 (colsum_kernel): for every scored key j < C-w,
//     a_j = (1/G) sum_rows exp2(l_rj*log2(e) - lse2_r),
//     a fixed-order reduction with no float atomics.
//
// Work split: workgroup = 8 waves; wave v holds row blocks v, v+8, v+16, ...
// (16 rows each) as MFMA A-fragments in registers, so a SIMD (waves v and
// v+4) covers a quarter of the rows. Each 64-key tile of K is staged once in
// LDS (the next tile is already in flight in registers) and read by all eight
// waves as B-fragments; blocks past the last row are skipped. MFMA
// 16x16x32 bf16 (or 8 x 16x16x4 f32 for fp32 inputs) accumulates in fp32.
// Output layout of a 16x16 MFMA: lane l holds rows 4*(l/16)+0..3 of key
// column l%16.
#include "device_common.h"
#include "mfma_frag.h"
#include "sgdkv_internal.h"

// Row blocks per wave the dispatch instantiates: at most 512 rows over all waves.
#define SGDKV_SCORE_WAVES_MAX_RBW (kMaxGroupRowsMacro / (16 * SGDKV_SCORE_WAVES))
#define kMaxGroupRowsMacro 512

namespace sgdkv {

// Shared pieces of both passes ------------------------------------------------
template <typename T, int D>
struct TileGeom {
  static constexpr int EB = elt_bytes<T>();
  static constexpr int RB = D * EB;           // bytes per key row
  static constexpr int LDS_STRIDE = RB + 16;  // padded row pitch: conflict-free 16-B fragment reads
  static constexpr int NC = D / 32;           // 32-wide k chunks
  static constexpr int V16 = RB / 16;         // 16-byte vectors per row
};

// K tile staging: keys [tile0, tile0+TILE) of this head travel global -> registers
// (issued one tile ahead) -> LDS. Keys past the end of the head read as zeros.
template <typename T, int D, int TILE>
struct KeyStage {
  using G = TileGeom<T, D>;
  static constexpr int N = (TILE * G::V16) / kScoreBlock;  // 16-byte vectors per thread
  static_assert(N >= 1 && (TILE * G::V16) % kScoreBlock == 0, "tile must split evenly");
  u32x4 r[N];
  __device__ __forceinline__ void load(rsrc_t kr, int64_t tile0) {
#pragma unroll
    for (int u = 0; u < N; ++u) {
      const int vi = threadIdx.x + u * kScoreBlock;
      const int row = vi / G::V16, c16 = vi % G::V16;
      r[u] = ld128(kr, (uint32_t)((tile0 + row) * G::RB + c16 * 16));
    }
  }
  __device__ __forceinline__ void store(char* ktile) const {
#pragma unroll
    for (int u = 0; u < N; ++u) {
      const int vi = threadIdx.x + u * kScoreBlock;
      const int row = vi / G::V16, c16 = vi % G::V16;
      *reinterpret_cast<u32x4*>(ktile + row * G::LDS_STRIDE + c16 * 16) = r[u];
    }
  }
};

template <typename T, int D, int RBW>
__device__ __forceinline__ void load_group_queries(const CompressArgs& a, int b, int h, int wid,
                                                   int lane, Frag<T> (&qa)[RBW][D / 32]) {
  using G = TileGeom<T, D>;
  const T* qbase = static_cast<const T*>(a.q_win) + ((int64_t)(b * a.Hq + h * a.G) * a.w) * D;
  const rsrc_t qr = make_rsrc(qbase, (uint64_t)a.R * G::RB);
  const int lr = lane & 15, lg = lane >> 4;
#pragma unroll
  for (int j = 0; j < RBW; ++j) {
    const int row = (wid + kScoreWaves * j) * 16 + lr;  // rows >= R read as zeros
#pragma unroll
    for (int c = 0; c < G::NC; ++c)
      qa[j][c] = gload_frag<T>(qr, (uint32_t)(row * G::RB + (32 * c + 8 * lg) * G::EB));
  }
}

// Per-tile compute -----------------------------------------------------------
//
// A tile of 16-key subtiles (64 keys for pass 2, 128 for pass 1) is one branch-free rolling
// pipeline: while subtile t's logits go through the vector ALU (one fma, one
// exp2, one add per logit), the MFMAs of subtile t+1 run on the matrix core and
// the key fragments of subtile t+2 are read from LDS. The MFMAs of each
// subtile are independent accumulator chains, one per row block.
template <typename T, int D, int NB>
__device__ __forceinline__ void subtile_mfma(const Frag<T> (&qa)[NB > 0 ? NB : 1][D / 32],
                                             const Frag<T> (&kb)[D / 32], f32x4 (&acc)[NB > 0 ? NB : 1]) {
#pragma unroll
  for (int c = 0; c < D / 32; ++c)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[j] = mma(qa[j][c], kb[c], c == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : acc[j]);
}

template <typename T, int D>
__device__ __forceinline__ void subtile_frags(const char* ktile, int t, int lr, int lg, Frag<T> (&kb)[D / 32]) {
  using G = TileGeom<T, D>;
#pragma unroll
  for (int c = 0; c < G::NC; ++c)
    kb[c] = lds_frag<T>(ktile, (uint32_t)((16 * t + lr) * G::LDS_STRIDE + (32 * c + 8 * lg) * G::EB));
}

// Runs op(t, acc_of_subtile_t) for the TILE/16 subtiles of the staged tile.
template <typename T, int D, int NB, int TILE, typename Op>
__device__ __forceinline__ void tile_pipeline(const char* ktile, int lr, int lg,
                                              const Frag<T> (&qa)[NB > 0 ? NB : 1][D / 32], Op&& op) {
  constexpr int NBX = NB > 0 ? NB : 1;
  constexpr int NT = TILE / 16;
  Frag<T> kb[2][D / 32];
  f32x4 acc[2][NBX];
  subtile_frags<T, D>(ktile, 0, lr, lg, kb[0]);
  subtile_frags<T, D>(ktile, 1, lr, lg, kb[1]);
  subtile_mfma<T, D, NB>(qa, kb[0], acc[0]);
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    if (t + 1 < NT) subtile_mfma<T, D, NB>(qa, kb[(t + 1) & 1], acc[(t + 1) & 1]);
    if (t + 2 < NT) subtile_frags<T, D>(ktile, t + 2, lr, lg, kb[t & 1]);
    op(t, acc[t & 1]);
  }
  // schedule: subtile 0's MFMAs, then the later MFMAs spread one per 3 vector instructions
#pragma unroll
  for (int i = 0; i < NB * (D / 32); ++i) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
#pragma unroll
  for (int i = 0; i < (NT - 1) * NB * (D / 32); ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);
  }
}

// Pass 1: per-chunk partial log-sum-exp of every window row -------------------
//
// Each lane keeps, for each of its 4*NB row slots, a reference m and a sum
// s = sum 2^(y - m) over the keys it has seen (y = logit * log2 e). Within a
// tile m is fixed, so each logit costs one fma, one exp2 and one add. After
// the tile, if any slot's sum left [0, 2^96] (a logit more than ~96 above its
// reference, +inf, or the +inf that m = -inf produces on a slot's first
// tile), the tile is redone for the whole wave from the saved sums with the
// exact online update (two exp2 per logit, m = running max). This happens on
// the first tile of a chunk, on tiles of the causal window block, and after
// rare large jumps. Padded rows (past R) start at m = 0 and are never stored.
template <typename T, int D, int NB, int TILE>
__device__ __forceinline__ void lse_exact_tile(const char* ktile, int lr, int lg, int wid, int w, int64_t tile0,
                                               int64_t vis0, const Frag<T> (&qa)[NB > 0 ? NB : 1][D / 32],
                                               float c2, float (&m)[NB > 0 ? NB : 1][4],
                                               float (&s)[NB > 0 ? NB : 1][4]) {
  constexpr int NBX = NB > 0 ? NB : 1;
  const bool masked = tile0 + TILE > vis0;
#pragma unroll 1
  for (int t = 0; t < TILE / 16; ++t) {
    Frag<T> kb[D / 32];
    subtile_frags<T, D>(ktile, t, lr, lg, kb);
    f32x4 acc[NBX];
    subtile_mfma<T, D, NB>(qa, kb, acc);
    const int64_t dk64 = tile0 + 16 * t + lr - vis0;
    const int dk = dk64 < -(1 << 30) ? -(1 << 30) : (int)dk64;
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int wi = ((wid + kScoreWaves * j) * 16 + 4 * lg + i) % w;  // window index of the row
        const float y = (masked && dk > wi) ? -INFINITY : acc[j][i] * c2;
        const float mn = fmaxf(m[j][i], y);
        if (mn != -INFINITY) {
          s[j][i] = s[j][i] * fast_exp2(m[j][i] - mn) + fast_exp2(y - mn);
          m[j][i] = mn;
        }
      }
  }
}

template <typename T, int D, int NB, int TILE>
__device__ __forceinline__ void lse_tile(const char* ktile, int lr, int lg, int wid, int w, int64_t tile0,
                                         int64_t vis0, const Frag<T> (&qa)[NB > 0 ? NB : 1][D / 32], float c2,
                                         float (&m)[NB > 0 ? NB : 1][4], float (&s)[NB > 0 ? NB : 1][4]) {
  constexpr int NBX = NB > 0 ? NB : 1;
  if (tile0 + TILE > vis0) {  // uniform: the tile reaches the causal window block
    lse_exact_tile<T, D, NB, TILE>(ktile, lr, lg, wid, w, tile0, vis0, qa, c2, m, s);
    return;
  }
  float s0[NBX][4];
#pragma unroll
  for (int j = 0; j < NBX; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) s0[j][i] = s[j][i];
  tile_pipeline<T, D, NB, TILE>(ktile, lr, lg, qa, [&](int, const f32x4(&acc)[NBX]) {
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) s[j][i] += fast_exp2(fmaf(acc[j][i], c2, -m[j][i]));
  });
  bool bad = false;
#pragma unroll
  for (int j = 0; j < NB; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) bad |= !(s[j][i] <= 7.9228162514264338e28f);  // 2^96; catches inf and NaN
  if (__any(bad)) {
#pragma unroll
    for (int j = 0; j < NBX; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) s[j][i] = s0[j][i];
    lse_exact_tile<T, D, NB, TILE>(ktile, lr, lg, wid, w, tile0, vis0, qa, c2, m, s);
  }
}

template <typename T, int D, int NB>
__device__ void lse_chunk(const CompressArgs& a, char* ktile, int seg, int wid, int lane,
                          const Frag<T> (&qa)[NB > 0 ? NB : 1][D / 32], const rsrc_t& kr, int64_t key0,
                          int64_t key_end) {
  constexpr int NBX = NB > 0 ? NB : 1;
  const int lr = lane & 15, lg = lane >> 4;
  const int64_t vis0 = a.C - a.w;  // the row with window index i sees key j iff j - vis0 <= i
  float m[NBX][4], s[NBX][4];
#pragma unroll
  for (int j = 0; j < NBX; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = (wid + kScoreWaves * j) * 16 + 4 * lg + i;
      m[j][i] = row < a.R ? -INFINITY : 0.f;  // a padded row must not force the exact path
      s[j][i] = 0.f;
    }
  const float c2 = a.c2;
  KeyStage<T, D, kLseTile> stage;
  stage.load(kr, key0);
  for (int64_t tile0 = key0; tile0 < key_end; tile0 += kLseTile) {
    __syncthreads();
    stage.store(ktile);
    __syncthreads();
    if (tile0 + kLseTile < key_end) stage.load(kr, tile0 + kLseTile);
    lse_tile<T, D, NB, kLseTile>(ktile, lr, lg, wid, a.w, tile0, vis0, qa, c2, m, s);
  }
  // Combine the 16 lanes (keys) of each row, then store (m, s) for the row.
  const int chunk = blockIdx.x;
  float* part = a.lse_part + ((int64_t)seg * a.n_lse_chunks + chunk) * a.R * 2;
  const rsrc_t pr = make_rsrc(part, (uint64_t)a.R * 2 * sizeof(float));
#pragma unroll
  for (int j = 0; j < NB; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float mm = m[j][i], ss = s[j][i];
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) {
        const float mo = __shfl_xor(mm, o, 64);
        const float so = __shfl_xor(ss, o, 64);
        const float mn = fmaxf(mm, mo);
        const float e1 = (mm == -INFINITY) ? 0.f : fast_exp2(mm - mn);
        const float e2 = (mo == -INFINITY) ? 0.f : fast_exp2(mo - mn);
        ss = ss * e1 + so * e2;
        mm = mn;
      }
      const int row = (wid + kScoreWaves * j) * 16 + 4 * lg + i;
      if (lr == 0 && row < a.R) {
        stf(pr, (uint32_t)(row * 8), mm);
        stf(pr, (uint32_t)(row * 8 + 4), ss);
      }
    }
}

template <typename T, int D, int RBW>
__global__ __launch_bounds__(kScoreBlock, 1) void lse_kernel(CompressArgs a) {
  using G = TileGeom<T, D>;
  __shared__ __attribute__((aligned(16))) char ktile[kLseTile * G::LDS_STRIDE];
  const int seg = blockIdx.y;
  const int b = seg / a.Hkv, h = seg % a.Hkv;
  const int64_t key0 = (int64_t)blockIdx.x * a.score_chunk;
  if (key0 >= a.C) return;
  const int64_t key_end = key0 + a.score_chunk < a.C ? key0 + a.score_chunk : a.C;
  const int tid = threadIdx.x, wid = tid >> 6, lane = tid & 63;
  const rsrc_t kr = make_rsrc(static_cast<const T*>(a.k) + (int64_t)seg * a.C * D, (uint64_t)a.C * G::RB);
  Frag<T> qa[RBW][G::NC];
  load_group_queries<T, D, RBW>(a, b, h, wid, lane, qa);
  // blocks this wave owns: RBW or RBW-1 (uniform per wave)
  const int nrb = (a.R + 15) / 16;
  if (wid + kScoreWaves * (RBW - 1) < nrb) {
    lse_chunk<T, D, RBW>(a, ktile, seg, wid, lane, qa, kr, key0, key_end);
  } else {
    Frag<T> qb[RBW > 1 ? RBW - 1 : 1][G::NC];
#pragma unroll
    for (int j = 0; j < RBW - 1; ++j)
#pragma unroll
      for (int c = 0; c < G::NC; ++c) qb[j][c] = qa[j][c];
    lse_chunk<T, D, RBW - 1>(a, ktile, seg, wid, lane, qb, kr, key0, key_end);
  }
}

// Merge the per-chunk partials of every window row in fp64: one wave per row,
// lanes stride over the chunks, fixed-order shuffle trees for max and sum.
__global__ __launch_bounds__(kBlock) void lse_merge_kernel(CompressArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t idx = (int64_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  const int64_t nrows = (int64_t)a.B * a.Hkv * a.R;
  if (idx >= nrows) return;  // uniform per wave
  const int64_t seg = idx / a.R, row = idx % a.R;
  const float* part = a.lse_part + (seg * a.n_lse_chunks) * a.R * 2;
  const rsrc_t pr = make_rsrc(part, (uint64_t)a.n_lse_chunks * a.R * 2 * sizeof(float));
  float mx = -INFINITY;
  for (int c = lane; c < a.n_lse_chunks; c += 64)
    mx = fmaxf(mx, ldf(pr, (uint32_t)(((int64_t)c * a.R + row) * 8)));
  mx = wave_max(mx);
  double sum = 0.0;
  if (mx != -INFINITY) {
    for (int c = lane; c < a.n_lse_chunks; c += 64) {
      const float mc = ldf(pr, (uint32_t)(((int64_t)c * a.R + row) * 8));
      const float sc = ldf(pr, (uint32_t)(((int64_t)c * a.R + row) * 8 + 4));
      if (mc != -INFINITY) sum += (double)sc * exp2((double)mc - (double)mx);
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) sum += __shfl_xor(sum, o, 64);
  if (lane == 0) {
    const float lse2 = (mx == -INFINITY || !(sum > 0.0)) ? -INFINITY : (float)((double)mx + log2(sum));
    const rsrc_t lr = make_rsrc(a.lse2, (uint64_t)nrows * sizeof(float));
    stf(lr, (uint32_t)(idx * 4), lse2);
  }
}

// Pass 2: window-summed probabilities of every scored key --------------------
template <typename T, int D, int NB>
__device__ void colsum_chunk(const CompressArgs& a, char* ktile, float (*red)[kColTile], int seg, int wid,
                             int lane, const Frag<T> (&qa)[NB > 0 ? NB : 1][D / 32], const rsrc_t& kr,
                             int64_t key0, int64_t key_end) {
  constexpr int NBX = NB > 0 ? NB : 1;
  const int tid = threadIdx.x;
  const int lr = lane & 15, lg = lane >> 4;
  // -lse2 of this lane's row slots; rows past R get -inf so they add exp2(-inf) = 0
  const uint64_t nl = (uint64_t)a.B * a.Hkv * a.R;
  const bool natural = a.window_lse != nullptr;
  const rsrc_t lr2 = make_rsrc(natural ? (const void*)a.window_lse : (const void*)a.lse2, nl * sizeof(float));
  float nlse[NBX][4];
#pragma unroll
  for (int j = 0; j < NBX; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = (wid + kScoreWaves * j) * 16 + 4 * lg + i;
      float l = ldf(lr2, (uint32_t)(((int64_t)seg * a.R + row) * 4));
      if (natural) l *= 1.44269504088896340736f;
      nlse[j][i] = row < a.R ? -l : -INFINITY;
    }
  const float c2 = a.c2;
  const rsrc_t cr = make_rsrc(a.colsum + (int64_t)seg * a.n_scored, (uint64_t)a.n_scored * 4);

  KeyStage<T, D, kColTile> stage;
  stage.load(kr, key0);
  for (int64_t tile0 = key0; tile0 < key_end; tile0 += kColTile) {
    __syncthreads();
    stage.store(ktile);
    __syncthreads();
    if (tile0 + kColTile < key_end) stage.load(kr, tile0 + kColTile);
    tile_pipeline<T, D, NB, kColTile>(ktile, lr, lg, qa, [&](int t, const f32x4(&acc)[NBX]) {
      // four independent partial sums (one per row slot) keep the add chains short
      float pp[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < NB; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) pp[i] += fast_exp2(fmaf(acc[j][i], c2, nlse[j][i]));
      float p = (pp[0] + pp[1]) + (pp[2] + pp[3]);
      p += __shfl_xor(p, 16, 64);
      p += __shfl_xor(p, 32, 64);
      red[wid][16 * t + lr] = p;  // all four lane groups hold the same value
    });
    __syncthreads();
    if (tid < kColTile) {
      const int64_t key = tile0 + tid;
      if (key < key_end) {
        float v = red[0][tid];
#pragma unroll
        for (int u = 1; u < kScoreWaves; ++u) v += red[u][tid];
        stf(cr, (uint32_t)(key * 4), v * a.inv_G);
      }
    }
  }
}

template <typename T, int D, int RBW>
__global__ __launch_bounds__(kScoreBlock, 1) void colsum_kernel(CompressArgs a) {
  using G = TileGeom<T, D>;
  __shared__ __attribute__((aligned(16))) char ktile[kColTile * G::LDS_STRIDE];
  __shared__ float red[kScoreWaves][kColTile];
  const int seg = blockIdx.y;
  const int b = seg / a.Hkv, h = seg % a.Hkv;
  const int64_t key0 = (int64_t)blockIdx.x * a.score_chunk;
  if (key0 >= a.n_scored) return;
  const int64_t key_end = key0 + a.score_chunk < a.n_scored ? key0 + a.score_chunk : a.n_scored;
  const int tid = threadIdx.x, wid = tid >> 6, lane = tid & 63;
  const rsrc_t kr = make_rsrc(static_cast<const T*>(a.k) + (int64_t)seg * a.C * D, (uint64_t)a.C * G::RB);
  Frag<T> qa[RBW][G::NC];
  load_group_queries<T, D, RBW>(a, b, h, wid, lane, qa);
  const int nrb = (a.R + 15) / 16;
  if (wid + kScoreWaves * (RBW - 1) < nrb) {
    colsum_chunk<T, D, RBW>(a, ktile, red, seg, wid, lane, qa, kr, key0, key_end);
  } else {
    Frag<T> qb[RBW > 1 ? RBW - 1 : 1][G::NC];
#pragma unroll
    for (int j = 0; j < RBW - 1; ++j)
#pragma unroll
      for (int c = 0; c < G::NC; ++c) qb[j][c] = qa[j][c];
    colsum_chunk<T, D, RBW - 1>(a, ktile, red, seg, wid, lane, qb, kr, key0, key_end);
  }
}

// Host-side dispatch ----------------------------------------------------------
template <typename T, int D, int RBW>
static hipError_t launch_scores_t(const CompressArgs& a, hipStream_t st) {
  const dim3 sblk(kScoreBlock);
  if (a.window_lse == nullptr) {
    SGDKV_LAUNCH("score_lse", (lse_kernel<T, D, RBW>), dim3(a.n_lse_chunks, a.B * a.Hkv), sblk, st, a);
    const int64_t nrows = (int64_t)a.B * a.Hkv * a.R;
    const int64_t rows_per_block = kBlock / 64;
    SGDKV_LAUNCH("lse_merge", lse_merge_kernel, dim3((unsigned)((nrows + rows_per_block - 1) / rows_per_block)),
                 dim3(kBlock), st, a);
  }
  if (a.n_col_chunks > 0)
    SGDKV_LAUNCH("score_colsum", (colsum_kernel<T, D, RBW>), dim3(a.n_col_chunks, a.B * a.Hkv), sblk, st, a);
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t launch_scores_d(const CompressArgs& a, hipStream_t st) {
  const int nrb = (a.R + 15) / 16;
  const int rbw = (nrb + kScoreWaves - 1) / kScoreWaves;
  switch (rbw) {
    case 1: return launch_scores_t<T, D, 1>(a, st);
    case 2: return launch_scores_t<T, D, 2>(a, st);
    case 3: return launch_scores_t<T, D, 3>(a, st);
    case 4: return launch_scores_t<T, D, 4>(a, st);
#if SGDKV_SCORE_WAVES_MAX_RBW > 4
    case 5: return launch_scores_t<T, D, 5>(a, st);
    case 6: return launch_scores_t<T, D, 6>(a, st);
    case 7: return launch_scores_t<T, D, 7>(a, st);
    case 8: return launch_scores_t<T, D, 8>(a, st);
#endif
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_scores(const CompressArgs& a, hipStream_t st) {
  if (a.dtype == 1) {
    if (a.D == 128) return launch_scores_d<__bf16, 128>(a, st);
    if (a.D == 64) return launch_scores_d<__bf16, 64>(a, st);
  } else {
    if (a.D == 128) return launch_scores_d<float, 128>(a, st);
    if (a.D == 64) return launch_scores_d<float, 64>(a, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace sgdkv
