// Observation-window scoring for SGD-KV token selection (gfx950).
//
// Token selection keeps, inside each KV head's budget, the keys with the
// largest cumulative attention of a final observation window (SGD-KV
// Sec. 3.3, last paragraph, SnapKV-style; Sec. 5 window placements). Window
// row i of query head q sits at prompt position P0+i (P0 = C-w for the
// Query-Aware window) and attends causally to keys 0..P0+i. For each KV head
// the G*w rows of its query group are one dense block R x d, so the logits of
// a key tile are an R x 16 MFMA product.
//
//   pass 1 (lse_kernel + lse_merge_kernel): base-2 log-sum-exp of every
//     window row over its causal keys. Each workgroup covers one chunk of
//     keys (about one workgroup per CU per launch) and leaves per-row partials
//     (m, s); the merge combines the chunks in a fixed order, in fp64.
//   pass 2 (colsum_kernel): for every scored key j < P0,
//     a_j = (1/G) sum_rows exp2(l_rj*log2(e) - lse2_r) (group mean; the Ipt.
//     aggregations below weight or pick rows), a fixed-order reduction with
//     no float atomics.
//
// Work split: workgroup = 8 waves; wave v holds row blocks v, v+8, v+16, ...
// (16 rows each) as MFMA A-fragments in registers, so a SIMD (waves v and
// v+4) covers a quarter of the rows. A workgroup holds at most 512 rows; a
// KV head with more window rows (G*w > 512, e.g. the 128-token window of the
// paper's main setting with GQA groups of 7 or 8) splits them over several
// workgroups per key chunk (grid z = row split). Pass 1 partials are per row
// anyway; pass 2 then leaves one column-sum partial per split, which the
// pooling pass adds (or, for Ipt. max, maximises) in split order. Each key tile (128 keys; 64 in pass 2
// for fp32 keys) is staged once in LDS and read by all eight waves as B-fragments;
// blocks past the last row are skipped. MFMA 16x16x32 bf16 (or 8 x 16x16x4
// f32 for fp32 inputs) accumulates in fp32.
// Output layout of a 16x16 MFMA: lane l holds rows 4*(l/16)+0..3 of key
// column l%16.
#include "device_common.h"
#include "mfma_frag.h"
#include "sgdkv_internal.h"
#include "segment_init.h"

// Row blocks per wave the dispatch instantiates: at most 512 rows (one row split) over all waves.
#define SGDKV_SCORE_WAVES_MAX_RBW (kMaxSplitRowsMacro / (16 * SGDKV_SCORE_WAVES))
#define kMaxSplitRowsMacro 512

namespace sgdkv {

// Shared pieces of both passes ------------------------------------------------
template <typename T>
constexpr int col_tile() {
  return sizeof(T) == 2 ? kColTileBf16 : kColTileF32;
}

template <typename T, int D>
struct TileGeom {
  static constexpr int EB = elt_bytes<T>();
  static constexpr int RB = D * EB;           // bytes per key row
  static constexpr int LDS_STRIDE = RB + 32;  // padded row pitch: 16-B fragment reads free of bank conflicts (measured)
  static constexpr int NC = D / 32;           // 32-wide k chunks
  static constexpr int V16 = RB / 16;         // 16-byte vectors per row
};

// K tile staging: keys [tile0, tile0+TILE) of this head travel global -> registers
// (issued one tile ahead) -> LDS. Keys past the end of the head read as zeros.
template <typename T, int D, int TILE>
struct KeyStage {
  using G = TileGeom<T, D>;
  static constexpr int TOT = TILE * G::V16;                        // 16-byte vectors per tile
  static constexpr int N = (TOT + kScoreBlock - 1) / kScoreBlock;  // per thread
  static constexpr bool ALL = TOT >= kScoreBlock;                  // every thread moves N vectors
  static_assert(TOT % kScoreBlock == 0 || !ALL, "tile must split evenly");
  u32x4 r[N];
  __device__ __forceinline__ void load(rsrc_t kr, int64_t tile0) {
    if (ALL || (int)threadIdx.x < TOT) {
#pragma unroll
      for (int u = 0; u < N; ++u) {
        const int vi = threadIdx.x + u * kScoreBlock;
        const int row = vi / G::V16, c16 = vi % G::V16;
        r[u] = ld128(kr, (uint32_t)((tile0 + row) * G::RB + c16 * 16));
      }
    }
  }
  __device__ __forceinline__ void store(char* ktile) const {
    if (ALL || (int)threadIdx.x < TOT) {
#pragma unroll
      for (int u = 0; u < N; ++u) {
        const int vi = threadIdx.x + u * kScoreBlock;
        const int row = vi / G::V16, c16 = vi % G::V16;
        *reinterpret_cast<u32x4*>(ktile + row * G::LDS_STRIDE + c16 * 16) = r[u];
      }
    }
  }
};

// Row block of slot j of wave wid: blocks wid, wid+8, ... (interleaved), or, with HW (head
// waves), blocks wid*RBW .. wid*RBW+RBW-1, so that the rows of a wave belong to one query head
// when w is a multiple of 16*RBW. Balanced head waves (bal: seven heads of one wave each, the
// group size of a 28/4-head model): the last wave, which would hold no rows, takes the last
// block of the heads of waves 4-6 (slots 0-2), so that each SIMD (waves s and s+4) carries
// 2*RBW - 1 blocks instead of 2*RBW on three SIMDs and RBW on the fourth.
constexpr int kBalFirstWave = kScoreWaves / 2;  // heads of waves 4-6 lend their last block
template <int RBW, bool HW>
__device__ __forceinline__ int row_block(int wid, int j, bool bal = false) {
  if (HW && bal && wid == kScoreWaves - 1) return (kBalFirstWave + j) * RBW + RBW - 1;
  return HW ? wid * RBW + j : wid + kScoreWaves * j;
}

// Window rows [r0, r0 + nrows) of KV head h (one row split) as A fragments.
template <typename T, int D, int RBW, bool HW = false>
__device__ __forceinline__ void load_group_queries(const CompressArgs& a, int b, int h, int r0, int nrows, int wid,
                                                   int lane, Frag<T> (&qa)[RBW][D / 32], bool bal = false) {
  using G = TileGeom<T, D>;
  const T* qbase = static_cast<const T*>(a.q_win) + ((int64_t)(b * a.Hq + h * a.G) * a.w + r0) * D;
  const rsrc_t qr = make_rsrc(qbase, (uint64_t)nrows * G::RB);
  const int lr = lane & 15, lg = lane >> 4;
#pragma unroll
  for (int j = 0; j < RBW; ++j) {
    const int row = row_block<RBW, HW>(wid, j, bal) * 16 + lr;  // rows >= nrows read as zeros
#pragma unroll
    for (int c = 0; c < G::NC; ++c)
      qa[j][c] = gload_frag<T>(qr, (uint32_t)(row * G::RB + (32 * c + 8 * lg) * G::EB));
  }
}

// Chunk pipeline --------------------------------------------------------------
//
// A workgroup streams the key tiles of its chunk through two LDS buffers and
// the MFMAs as one rolling pipeline. In step s of tile t a wave issues the
// MFMAs of the next subtile (16 keys), reads the key fragments of the subtile
// after that from LDS, and hands the logits of subtile s to the vector ALU.
// Tile t+1 goes into the other buffer at the start of tile t (its global loads
// were issued one tile earlier), and the tile's single barrier, two subtiles
// before its end, makes that buffer readable; the buffer written at the start
// of tile t was last read before the barrier of tile t-1. The MFMAs of the
// subtile after the chunk's last one run on whatever keys follow (zeros past
// the head) and are discarded. REV streams the chunk's tiles last to first
// (step t covers tile ntiles-1-t; the steps after the last read zeros). On
// gfx950 a wave's own MFMAs and vector instructions issue one after the other,
// and exp2 overlaps little with the MFMAs of the SIMD's other wave; the two
// waves of a SIMD mainly hide each other's latencies.
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

// Hooks: begin(acc) once with the logits of the chunk's first subtile (before
// any sub call); sub(t, s, acc) per subtile; at_barrier(t) right after tile t's
// barrier; end_tile(t) after tile t's last subtile.
template <typename T, int D, int NB, int TILE, bool REV = false, typename Begin, typename Sub, typename AtBarrier,
          typename EndTile>
__device__ __forceinline__ void chunk_pipeline(char* kbuf, const rsrc_t& kr, int64_t key0, int64_t C, int64_t ntiles,
                                               int lr, int lg, const Frag<T> (&qa)[NB > 0 ? NB : 1][D / 32],
                                               Begin&& begin, Sub&& sub, AtBarrier&& at_barrier, EndTile&& end_tile) {
  using G = TileGeom<T, D>;
  constexpr int NBX = NB > 0 ? NB : 1;
  constexpr int S = TILE / 16;
  constexpr int BUF = TILE * G::LDS_STRIDE;
  static_assert(S >= 4 && S % 2 == 0, "tile geometry");
  // keys past the head read as zeros; the clamp keeps byte offsets below 4 GiB
  auto tile_key = [&](int64_t t) {
    const int64_t k = REV ? (t < ntiles ? key0 + (ntiles - 1 - t) * TILE : C) : key0 + t * TILE;
    return k < C ? k : C;
  };
  KeyStage<T, D, TILE> stage;
  stage.load(kr, tile_key(0));
  stage.store(kbuf);
  stage.load(kr, tile_key(1));
  __syncthreads();
  Frag<T> kb[2][D / 32];
  f32x4 acc[2][NBX];
  subtile_frags<T, D>(kbuf, 0, lr, lg, kb[0]);
  subtile_frags<T, D>(kbuf, 1, lr, lg, kb[1]);
  subtile_mfma<T, D, NB>(qa, kb[0], acc[0]);
  begin(acc[0]);
  for (int64_t t = 0; t < ntiles; ++t) {
    const char* buf = kbuf + (t & 1) * BUF;
    char* nbuf = kbuf + ((t + 1) & 1) * BUF;
#pragma unroll
    for (int s = 0; s < S; ++s) {
      if (s == 0) {
        stage.store(nbuf);
        stage.load(kr, tile_key(t + 2));
      }
      if (s == S - 2) {
        __syncthreads();
        at_barrier(t);
      }
      subtile_mfma<T, D, NB>(qa, kb[(s + 1) & 1], acc[(s + 1) & 1]);
      if (s + 2 < S)
        subtile_frags<T, D>(buf, s + 2, lr, lg, kb[s & 1]);
      else
        subtile_frags<T, D>(nbuf, s + 2 - S, lr, lg, kb[s & 1]);
      sub(t, s, acc[s & 1]);
    }
    end_tile(t);
  }
}

// Pass 1: per-chunk partial log-sum-exp of every window row -------------------
//
// Each lane keeps, for each of its 4*NB row slots, a reference m and a sum
// s = sum 2^(y - m) over the keys it has seen (y = logit * log2 e). The tiles
// of the chunk that every window row sees in full run through the pipeline
// with m fixed at the row's largest logit among the chunk's first 16 keys, so
// each logit costs one fma, one exp2 and one add and the loop has no branch.
// A sum can only overflow if a later logit exceeds that maximum by about 100
// (base 2); the chunk's sums are checked once at its end and, if any left
// [0, 2^122] (inf and NaN included), the whole chunk is recomputed with the
// exact online update (two exp2 per logit, m = running max), reading the keys
// from global memory. The bound leaves room for the 16 lanes of a row, which
// share the reference and are then added as they are: 16 * 2^122 = 2^126 stays
// finite. The tiles that reach the window block (causal mask) or
// pass the end of the head always take that exact path. Padded rows (past R)
// keep m = 0.
template <typename T, int D, int NB, int TILE>
__device__ __forceinline__ void lse_exact_tile(const rsrc_t& kr, int lr, int lg, int wid, int r0, int w, int64_t tile0,
                                            int64_t vis0, int64_t C, const Frag<T> (&qa)[NB > 0 ? NB : 1][D / 32],
                                            float c2, float (&m)[NB > 0 ? NB : 1][4],
                                            float (&s)[NB > 0 ? NB : 1][4]) {
  using G = TileGeom<T, D>;
  constexpr int NBX = NB > 0 ? NB : 1;
  const bool masked = tile0 + TILE > vis0;
  auto load = [&](int t, Frag<T>(&kb)[D / 32]) {
#pragma unroll
    for (int c = 0; c < G::NC; ++c)
      kb[c] = gload_frag<T>(kr, (uint32_t)((tile0 + 16 * t + lr) * G::RB + (32 * c + 8 * lg) * G::EB));
  };
  Frag<T> kn[D / 32];
  load(0, kn);
#pragma unroll 1
  for (int t = 0; t < TILE / 16; ++t) {
    Frag<T> kb[D / 32];
#pragma unroll
    for (int c = 0; c < G::NC; ++c) kb[c] = kn[c];
    load(t + 1 < TILE / 16 ? t + 1 : t, kn);  // the next subtile's keys are in flight during this one
    f32x4 acc[NBX];
    subtile_mfma<T, D, NB>(qa, kb, acc);
    const int64_t key = tile0 + 16 * t + lr;
    const int64_t dk64 = key < C ? key - vis0 : (int64_t)1 << 30;  // keys past the head: never visible
    const int dk = dk64 < -(1 << 30) ? -(1 << 30) : (dk64 > (1 << 30) ? (1 << 30) : (int)dk64);
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int wi = (r0 + (wid + kScoreWaves * j) * 16 + 4 * lg + i) % w;  // window index of the row
        const float y = (masked && dk > wi) ? -INFINITY : acc[j][i] * c2;
        const float mn = fmaxf(m[j][i], y);
        if (mn != -INFINITY) {
          s[j][i] = s[j][i] * fast_exp2(m[j][i] - mn) + fast_exp2(y - mn);
          m[j][i] = mn;
        }
      }
  }
}

template <typename T, int D, int NB>
__device__ void lse_chunk(const CompressArgs& a, char* kbuf, int seg, int chunk, int r0, int nrows, int wid,
                          int lane, const Frag<T> (&qa)[NB > 0 ? NB : 1][D / 32], const rsrc_t& kr, int64_t key0,
                          int64_t key_end) {
  constexpr int NBX = NB > 0 ? NB : 1;
  constexpr int TILE = kLseTile;
  const int lr = lane & 15, lg = lane >> 4;
  const int64_t vis0 = a.win0;  // the row with window index i sees key j iff j - vis0 <= i (and j < C)
  const float c2 = a.c2;
  float m[NBX][4], s[NBX][4];
  bool real[NBX][4];
  auto reset = [&]() {
#pragma unroll
    for (int j = 0; j < NBX; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        m[j][i] = real[j][i] ? -INFINITY : 0.f;  // a padded row must not force the exact path
        s[j][i] = 0.f;
      }
  };
#pragma unroll
  for (int j = 0; j < NBX; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) real[j][i] = (wid + kScoreWaves * j) * 16 + 4 * lg + i < nrows;
  reset();
  // whole tiles every row sees (keys below both the window block and the end of the head)
  const int64_t open_end = vis0 < a.C ? vis0 : a.C;
  const int64_t fast_end = key_end < open_end ? key_end : open_end;
  const int64_t nfast = fast_end > key0 ? (fast_end - key0) / TILE : 0;
  const int64_t ntiles = (key_end - key0 + TILE - 1) / TILE;
  if (nfast > 0) {
    chunk_pipeline<T, D, NB, TILE>(
        kbuf, kr, key0, a.C, nfast, lr, lg, qa,
        [&](const f32x4(&acc)[NBX]) {
#pragma unroll
          for (int j = 0; j < NB; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float mx = row16_max(acc[j][i] * c2);  // every lane of the 16-lane row takes part
              if (real[j][i]) m[j][i] = mx;
            }
        },
        [&](int64_t, int, const f32x4(&acc)[NBX]) {
#pragma unroll
          for (int j = 0; j < NB; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i) s[j][i] += fast_exp2(fmaf(acc[j][i], c2, -m[j][i]));
        },
        [&](int64_t) {}, [&](int64_t) {});
    bool bad = false;
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) bad |= !(s[j][i] <= 5.3169119831396635e36f);  // 2^122; catches inf and NaN
    if (__any(bad)) {
      reset();
      for (int64_t t = 0; t < nfast; ++t)
        lse_exact_tile<T, D, NB, TILE>(kr, lr, lg, wid, r0, a.w, key0 + t * TILE, vis0, a.C, qa, c2, m, s);
    }
  }
  for (int64_t t = nfast; t < ntiles; ++t)
    lse_exact_tile<T, D, NB, TILE>(kr, lr, lg, wid, r0, a.w, key0 + t * TILE, vis0, a.C, qa, c2, m, s);
  // Combine the 16 lanes (keys) of each row, then store (m, s) for the row.
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
      if (lr == 0 && row < nrows) {
        stf(pr, (uint32_t)((r0 + row) * 8), mm);
        stf(pr, (uint32_t)((r0 + row) * 8 + 4), ss);
      }
    }
}

template <typename T, int D, int RBW>
__global__ __launch_bounds__(kScoreBlock, 1) void lse_kernel(CompressArgs a) {
  using G = TileGeom<T, D>;
  __shared__ __attribute__((aligned(16))) char ktile[2 * kLseTile * G::LDS_STRIDE];
  const int seg = blockIdx.y;
  const int b = seg / a.Hkv, h = seg % a.Hkv;
  // the tail chunk (the causally masked tiles, on the exact path) goes first, then the uniform
  // chunks of keys every row sees; keys past the last window row's position are seen by no row
  const int chunk = (int)(gridDim.x - 1 - blockIdx.x);
  const int64_t vis_end = a.win0 + a.w < a.C ? a.win0 + a.w : a.C;
  int64_t key0, key_end;
  if (chunk < a.n_lse_head) {
    key0 = (int64_t)chunk * a.lse_chunk;
    key_end = key0 + a.lse_chunk < a.lse_tail0 ? key0 + a.lse_chunk : a.lse_tail0;
  } else {
    key0 = a.lse_tail0;
    key_end = vis_end;
  }
  if (key0 >= key_end) return;
  const int tid = threadIdx.x, wid = tid >> 6, lane = tid & 63;
  const int r0 = (int)blockIdx.z * a.lse_rs_rows;
  const int nrows = a.R - r0 < a.lse_rs_rows ? a.R - r0 : a.lse_rs_rows;
  const rsrc_t kr = make_rsrc(static_cast<const T*>(a.k) + (int64_t)seg * a.C * D, (uint64_t)a.C * G::RB);
  Frag<T> qa[RBW][G::NC];
  load_group_queries<T, D, RBW>(a, b, h, r0, nrows, wid, lane, qa);
  // blocks this wave owns: RBW or RBW-1 (uniform per wave)
  const int nrb = (nrows + 15) / 16;
  if (wid + kScoreWaves * (RBW - 1) < nrb) {
    lse_chunk<T, D, RBW>(a, ktile, seg, chunk, r0, nrows, wid, lane, qa, kr, key0, key_end);
  } else {
    Frag<T> qb[RBW > 1 ? RBW - 1 : 1][G::NC];
#pragma unroll
    for (int j = 0; j < RBW - 1; ++j)
#pragma unroll
      for (int c = 0; c < G::NC; ++c) qb[j][c] = qa[j][c];
    lse_chunk<T, D, RBW - 1>(a, ktile, seg, chunk, r0, nrows, wid, lane, qb, kr, key0, key_end);
  }
}

// Merge the per-chunk partials of every window row in fp64: 16 lanes per row (16 rows per
// workgroup of segment blockIdx.y), lane l taking chunks l, l+16, ...; the maximum of the chunk
// references over the 16 lanes, then each lane's rescaled sums in chunk order, and the 16 lane
// sums added in a fixed butterfly order. A row's lanes read neighbouring chunks' partials.
constexpr int kMergeLanes = 16;
__global__ __launch_bounds__(kBlock) void lse_merge_kernel(CompressArgs a) {
  const int64_t seg = blockIdx.y;
  const int lane = threadIdx.x % kMergeLanes;
  const int row = blockIdx.x * (kBlock / kMergeLanes) + threadIdx.x / kMergeLanes;
  const bool live = row < a.R;  // every lane takes part in the shuffles
  const int n = a.n_lse_chunks;
  const rsrc_t pr = make_rsrc(a.lse_part + seg * n * a.R * 2, (uint64_t)n * a.R * 2 * sizeof(float));
  auto off = [&](int c) { return (uint32_t)(((int64_t)c * a.R + row) * 8); };
  float mx = -INFINITY;
  if (live)
    for (int c = lane; c < n; c += kMergeLanes) mx = fmaxf(mx, ldf(pr, off(c)));
#pragma unroll
  for (int o = 1; o < kMergeLanes; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
  double sum = 0.0;
  if (live && mx != -INFINITY) {
    for (int c = lane; c < n; c += kMergeLanes) {
      const uint64_t ms = ld64(pr, off(c));
      const float mc = __uint_as_float((uint32_t)ms), sc = __uint_as_float((uint32_t)(ms >> 32));
      if (mc != -INFINITY) sum += (double)sc * exp2((double)mc - (double)mx);
    }
  }
#pragma unroll
  for (int o = 1; o < kMergeLanes; o <<= 1) sum += __shfl_xor(sum, o, 64);
  if (!live || lane != 0) return;
  const float lse2 = (mx == -INFINITY || !(sum > 0.0)) ? -INFINITY : (float)((double)mx + log2(sum));
  const rsrc_t lr = make_rsrc(a.lse2 + seg * a.R, (uint64_t)a.R * sizeof(float));
  stf(lr, (uint32_t)row * 4u, lse2);
}

// Pass 2: window-summed probabilities of every scored key --------------------
//
// Group aggregation. Row r of a KV head's window block belongs to query head
// g = r / w of the group. The group mean, Ipt. mean and Ipt. only sum every
// row with a weight (1, sigma_g, or 1 for the top-scored head and 0 for the
// others), folded into the exp2 argument as log2 of the weight, so they cost
// nothing extra. Ipt. max (MAXG) needs each query head's own column sum. With
// head waves (HW: a wave's row blocks are consecutive and lie in one query
// head, which needs w to be a multiple of 16*RBW) the waves sum their rows as
// for the group mean and the reduction adds the partials of each head's
// waves, weights them and takes the maximum. Otherwise the waves keep one
// partial per row block (16 rows of a single head when w is a multiple of
// 16), and the reduction adds each head's blocks the same way.
template <bool MAXG, bool HW>
constexpr bool block_partials() {
  return MAXG && !HW;
}
// Balanced head waves: the last wave keeps four lane-group partials for each of its three blocks,
// 12 rows instead of 4.
template <bool MAXG, bool HW, int RBW>
constexpr int bal_extra_rows() {
  return MAXG && HW && RBW == 4 ? 8 : 0;
}

// LDS layout of pass 2's column partials: three tiles in flight, each with RW partial rows of
// TILE columns per wave. A partial row is 16 banks further than the one before it and a wave's
// rows 16 banks further again, so that neither the four lane groups of a wave storing a subtile
// nor the four waves whose partials the reduction reads together meet in one bank.
template <typename T, int RW, int EXTRA = 0>
struct ColPartials {
  static constexpr int TILE = col_tile<T>();
  static constexpr int SL = TILE + 16;         // floats per partial row
  static constexpr int SW = RW * SL + 16;      // floats per wave
  static constexpr int ST = kScoreWaves * SW + EXTRA * SL;  // floats per tile (EXTRA more rows for the last wave)
  static constexpr int WORDS = 3 * ST;
  __device__ static constexpr int at(int t3, int wave, int r, int col) { return t3 * ST + wave * SW + r * SL + col; }
};

// MIXED: the wave's blocks belong to different heads (the last wave of the balanced head-wave
// layout): it leaves four lane-group partials per block, in rows 4j .. 4j+3 of its region.
template <typename T, int D, int NB, int RBW, bool MAXG, bool HW, bool MIXED = false>
__device__ void colsum_chunk(const CompressArgs& a, char* kbuf, float* red, float* qws, int seg, int r0, int nrows,
                             int wid, int lane,
                             const Frag<T> (&qa)[NB > 0 ? NB : 1][D / 32], const rsrc_t& kr, int64_t key0,
                             int64_t key_end, bool bal = false) {
  constexpr int NBX = NB > 0 ? NB : 1;
  constexpr int TILE = col_tile<T>();
  const int lr = lane & 15, lg = lane >> 4;
  const int h = seg % a.Hkv;
  // -lse2 (+ log2 of the row weight) of this lane's row slots; rows past R get -inf so they add 0
  const uint64_t nl = (uint64_t)a.B * a.Hkv * a.R;
  const bool natural = a.window_lse != nullptr;
  const bool weighted = !MAXG && a.agg != 0;
  const rsrc_t lr2 = make_rsrc(natural ? (const void*)a.window_lse : (const void*)a.lse2, nl * sizeof(float));
  float nlse[NBX][4];
#pragma unroll
  for (int j = 0; j < NBX; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = row_block<RBW, HW>(wid, j, bal) * 16 + 4 * lg + i;  // within the split
      float l = ldf(lr2, (uint32_t)(((int64_t)seg * a.R + r0 + row) * 4));
      if (natural) l *= 1.44269504088896340736f;
      const float lw = weighted && row < nrows ? a.qweight[h * a.G + (r0 + row) / a.w] : 0.f;
      nlse[j][i] = row < nrows ? lw - l : -INFINITY;
    }
  const float c2 = a.c2;
  const int nseg = a.B * a.Hkv;
  const rsrc_t cr = make_rsrc(a.colsum + ((int64_t)blockIdx.z * nseg + seg) * a.n_scored, (uint64_t)a.n_scored * 4);
  // The chunk's tiles go last to first: pass 1 streams about the same chunks first to last, so
  // the keys it read last, the ends of the chunks, are partly still in the last-level cache.
  // Each key's sum does not depend on the order, so neither does the result.
  const int64_t ntiles = (key_end - key0 + TILE - 1) / TILE;
  // Partials of tile t sit in red[t % 3]: written during tile t, complete at the barrier of
  // tile t+1, summed right after it, rewritten only after the barrier of tile t+2. Each
  // wave sums CPW columns: the LPC lanes of a column read the partials of PPL waves each
  // (one per lane group of the wave for the group mean), shuffles add them, and the first
  // CPW lanes store. Branch-free: a store that must not happen gets an
  // offset past the buffer, which the hardware drops.
  constexpr int CPW = TILE / kScoreWaves, LPC = 64 / CPW, PPL = kScoreWaves / LPC;
  static_assert(CPW <= 16 && 64 % CPW == 0 && PPL >= 1 && PPL * LPC == kScoreWaves, "reduction layout");
  const int rcol = CPW * wid + lane % CPW, rgrp = lane / CPW;
  constexpr bool BP = block_partials<MAXG, HW>();
  using CP = ColPartials<T, BP ? RBW : 4, bal_extra_rows<MAXG, HW, RBW>()>;
  // Ipt. max: the split's head weights go to LDS once (a global load in the per-tile reduction
  // would wait behind the key tiles in flight)
  if constexpr (MAXG) {
    const int g0 = r0 / a.w, ng = nrows / a.w;  // at most kMaxSplitRows / 16 heads
    if (wid == 0 && lane < ng) qws[lane] = a.qweight[h * a.G + g0 + lane];
    __syncthreads();
  }
  auto reduce = [&](int64_t t) {  // t may be -1: nothing is stored
    const float* r = red + CP::at((int)((uint32_t)(t + 3) % 3u), 0, 0, 0);
    float v = 0.f;
    if constexpr (MAXG && HW) {
      // the LPC lanes of a column take the split's heads in turn: add the four lane-group
      // partials of each of a head's w/(16*RBW) waves in wave order, weight, keep the maximum
      // (balanced layout: heads 4-6 then add the four lane-group partials of the block they lent
      // to the last wave)
      const int wph = a.w / (16 * RBW), ng = nrows / a.w;
      for (int g = rgrp; g < ng; g += LPC) {
        float sum = 0.f;
        for (int wv = g * wph; wv < (g + 1) * wph; ++wv)
#pragma unroll
          for (int q = 0; q < 4; ++q) sum += r[wv * CP::SW + q * CP::SL + rcol];
        if (bal && g >= kBalFirstWave) {
          const float* lent = r + (kScoreWaves - 1) * CP::SW + 4 * (g - kBalFirstWave) * CP::SL + rcol;
#pragma unroll
          for (int q = 0; q < 4; ++q) sum += lent[q * CP::SL];
        }
        v = fmaxf(v, qws[g] * sum);
      }
#pragma unroll
      for (int o = CPW; o < 16; o <<= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
      v = max_lane_groups(v);
    } else if constexpr (MAXG) {
      // the LPC lanes of a column take the split's heads in turn: sum a head's w/16 blocks
      // (block b sits with wave b % 8, slot b / 8), weight it, keep the maximum
      const int bph = a.w / 16, ng = nrows / a.w;
      for (int g = rgrp; g < ng; g += LPC) {
        float sum = 0.f;
        for (int bb = g * bph; bb < (g + 1) * bph; ++bb)
          sum += r[(bb % kScoreWaves) * CP::SW + (bb / kScoreWaves) * CP::SL + rcol];
        v = fmaxf(v, qws[g] * sum);
      }
#pragma unroll
      for (int o = CPW; o < 16; o <<= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
      v = max_lane_groups(v);
    } else {
      // the partials of every wave and lane group of the column, in a fixed order
#pragma unroll
      for (int k = 0; k < PPL; ++k)
#pragma unroll
        for (int g = 0; g < 4; ++g) v += r[(rgrp + LPC * k) * CP::SW + g * CP::SL + rcol];
#pragma unroll
      for (int o = CPW; o < 16; o <<= 1) v += __shfl_xor(v, o, 64);
      v = sum_lane_groups(v);
    }
    const int64_t key = key0 + (ntiles - 1 - t) * TILE + rcol;  // step t holds tile ntiles-1-t
    const bool store = t >= 0 && lane < CPW && key < key_end;
    stf(cr, store ? (uint32_t)(key * 4) : (uint32_t)(a.n_scored * 4), v * a.out_scale);
  };
  chunk_pipeline<T, D, NB, TILE, true>(
      kbuf, kr, key0, a.C, ntiles, lr, lg, qa, [](const f32x4(&)[NBX]) {},
      [&](int64_t t, int sub, const f32x4(&acc)[NBX]) {
        const int t3 = (int)((uint32_t)t % 3u);  // tiles of a chunk: far fewer than 2^32
        if constexpr (BP) {
          // one column partial per row block (a single query head's rows)
#pragma unroll
          for (int j = 0; j < NB; ++j) {
            const float p = (fast_exp2(fmaf(acc[j][0], c2, nlse[j][0])) + fast_exp2(fmaf(acc[j][1], c2, nlse[j][1]))) +
                            (fast_exp2(fmaf(acc[j][2], c2, nlse[j][2])) + fast_exp2(fmaf(acc[j][3], c2, nlse[j][3])));
            red[CP::at(t3, wid, j, 16 * sub + lr)] = sum_lane_groups(p);
          }
        } else if constexpr (MIXED) {
          // four lane-group partials per block (each block a different head's rows)
#pragma unroll
          for (int j = 0; j < NB; ++j) {
            const float p = (fast_exp2(fmaf(acc[j][0], c2, nlse[j][0])) + fast_exp2(fmaf(acc[j][1], c2, nlse[j][1]))) +
                            (fast_exp2(fmaf(acc[j][2], c2, nlse[j][2])) + fast_exp2(fmaf(acc[j][3], c2, nlse[j][3])));
            red[CP::at(t3, wid, 4 * j + lg, 16 * sub + lr)] = p;
          }
        } else {
          float p = 0.f;
          if constexpr (NB > 0) {
            // four independent partial sums (one per row slot) keep the add chains short
            float pp[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) pp[i] = fast_exp2(fmaf(acc[0][i], c2, nlse[0][i]));
#pragma unroll
            for (int j = 1; j < NB; ++j)
#pragma unroll
              for (int i = 0; i < 4; ++i) pp[i] += fast_exp2(fmaf(acc[j][i], c2, nlse[j][i]));
            p = (pp[0] + pp[1]) + (pp[2] + pp[3]);
          }
          red[CP::at(t3, wid, lg, 16 * sub + lr)] = p;  // one partial per lane group; the reduction adds them
        }
      },
      [&](int64_t t) { reduce(t - 1); }, [](int64_t) {});
  __syncthreads();
  reduce(ntiles - 1);
}

template <typename T, int D, int RBW, bool MAXG, bool HW>
__global__ __launch_bounds__(kScoreBlock, 1) void colsum_kernel(CompressArgs a) {
  using G = TileGeom<T, D>;
  __shared__ __attribute__((aligned(16))) char ktile[2 * col_tile<T>() * G::LDS_STRIDE];
  __shared__ __attribute__((aligned(16)))
  float red[ColPartials<T, block_partials<MAXG, HW>() ? RBW : 4, bal_extra_rows<MAXG, HW, RBW>()>::WORDS];
  __shared__ float qws[MAXG ? kMaxSplitRows / 16 : 1];  // Ipt. max: the row split's head weights
  const int seg = blockIdx.y;
  const int b = seg / a.Hkv, h = seg % a.Hkv;
  if (blockIdx.x == 0 && blockIdx.z == 0) init_segment(a, seg);  // histograms, offsets for the selection
  const int64_t key0 = (int64_t)blockIdx.x * a.score_chunk;
  if (key0 >= a.n_scored) return;
  const int64_t key_end = key0 + a.score_chunk < a.n_scored ? key0 + a.score_chunk : a.n_scored;
  const int tid = threadIdx.x, wid = tid >> 6, lane = tid & 63;
  const int r0 = (int)blockIdx.z * a.rs_rows;
  const int nrows = a.R - r0 < a.rs_rows ? a.R - r0 : a.rs_rows;
  const rsrc_t kr = make_rsrc(static_cast<const T*>(a.k) + (int64_t)seg * a.C * D, (uint64_t)a.C * G::RB);
  // balanced head waves: a split of seven heads of one wave each, four blocks per head (with
  // three blocks per head the busiest SIMD would carry six blocks either way)
  constexpr bool can_bal = MAXG && HW && RBW == 4;
  const bool bal = can_bal && nrows == 7 * a.w && a.w == 16 * RBW;
  Frag<T> qa[RBW][G::NC];
  load_group_queries<T, D, RBW, HW>(a, b, h, r0, nrows, wid, lane, qa, bal);
  const int nrb = (nrows + 15) / 16;
  if constexpr (HW) {
    // a row split holds whole heads of w/16 blocks, a multiple of RBW: each wave has all
    // RBW of its blocks or none (a wave without rows still stages keys and meets every barrier)
    if constexpr (can_bal) {
      if (bal && wid >= kBalFirstWave) {
        Frag<T> qb[3][G::NC];  // waves 4-6: their first three blocks; wave 7: the three lent blocks
#pragma unroll
        for (int j = 0; j < 3; ++j)
#pragma unroll
          for (int c = 0; c < G::NC; ++c) qb[j][c] = qa[j][c];
        if (wid == kScoreWaves - 1)
          colsum_chunk<T, D, 3, RBW, MAXG, HW, true>(a, ktile, red, qws, seg, r0, nrows, wid, lane, qb, kr, key0,
                                                     key_end, bal);
        else
          colsum_chunk<T, D, 3, RBW, MAXG, HW>(a, ktile, red, qws, seg, r0, nrows, wid, lane, qb, kr, key0, key_end,
                                               bal);
        return;
      }
    }
    // (every wave reduces some columns, so each needs to know the layout: bal goes to all)
    if (row_block<RBW, HW>(wid, 0) < nrb) {
      colsum_chunk<T, D, RBW, RBW, MAXG, HW>(a, ktile, red, qws, seg, r0, nrows, wid, lane, qa, kr, key0, key_end, bal);
    } else {
      Frag<T> qz[1][G::NC];  // never read: the wave has no row blocks
#pragma unroll
      for (int c = 0; c < G::NC; ++c) qz[0][c] = qa[0][c];
      colsum_chunk<T, D, 0, RBW, MAXG, HW>(a, ktile, red, qws, seg, r0, nrows, wid, lane, qz, kr, key0, key_end, bal);
    }
  } else if (wid + kScoreWaves * (RBW - 1) < nrb) {
    colsum_chunk<T, D, RBW, RBW, MAXG, HW>(a, ktile, red, qws, seg, r0, nrows, wid, lane, qa, kr, key0, key_end);
  } else {
    Frag<T> qb[RBW > 1 ? RBW - 1 : 1][G::NC];
#pragma unroll
    for (int j = 0; j < RBW - 1; ++j)
#pragma unroll
      for (int c = 0; c < G::NC; ++c) qb[j][c] = qa[j][c];
    colsum_chunk<T, D, RBW - 1, RBW, MAXG, HW>(a, ktile, red, qws, seg, r0, nrows, wid, lane, qb, kr, key0, key_end);
  }
}

// Host-side dispatch ----------------------------------------------------------
// Pass 1 (and its merge) with RBW row blocks per wave for its row split.
template <typename T, int D, int RBW>
static hipError_t launch_lse_t(const CompressArgs& a, hipStream_t st) {
  const dim3 sblk(kScoreBlock);
  SGDKV_LAUNCH("score_lse", (lse_kernel<T, D, RBW>), dim3(a.n_lse_chunks, a.B * a.Hkv, a.lse_n_rsplit), sblk, st, a);
  constexpr int rows_per_wg = kBlock / kMergeLanes;
  SGDKV_LAUNCH("lse_merge", lse_merge_kernel, dim3((unsigned)((a.R + rows_per_wg - 1) / rows_per_wg), a.B * a.Hkv),
               dim3(kBlock), st, a);
  return hipGetLastError();
}

// Pass 2 with RBW row blocks per wave for its row split.
template <typename T, int D, int RBW>
static hipError_t launch_colsum_t(const CompressArgs& a, hipStream_t st) {
  const dim3 sblk(kScoreBlock);
  if (a.n_col_chunks > 0) {
    const dim3 cgrid(a.n_col_chunks, a.B * a.Hkv, a.n_rsplit);
    if (a.agg == 1 && a.w % (16 * RBW) == 0)
      SGDKV_LAUNCH("score_colsum", (colsum_kernel<T, D, RBW, true, true>), cgrid, sblk, st, a);
    else if (a.agg == 1)
      SGDKV_LAUNCH("score_colsum", (colsum_kernel<T, D, RBW, true, false>), cgrid, sblk, st, a);
    else
      SGDKV_LAUNCH("score_colsum", (colsum_kernel<T, D, RBW, false, false>), cgrid, sblk, st, a);
  }
  return hipGetLastError();
}

// Row blocks per wave for a row split of `rows` rows (its largest split), as a template argument.
template <typename T, int D, template <typename, int, int> class L>
static hipError_t dispatch_rbw(int rows, const CompressArgs& a, hipStream_t st) {
  const int nrb = (rows + 15) / 16;
  switch ((nrb + kScoreWaves - 1) / kScoreWaves) {
    case 1: return L<T, D, 1>::run(a, st);
    case 2: return L<T, D, 2>::run(a, st);
    case 3: return L<T, D, 3>::run(a, st);
    case 4: return L<T, D, 4>::run(a, st);
#if SGDKV_SCORE_WAVES_MAX_RBW > 4
    case 5: return L<T, D, 5>::run(a, st);
    case 6: return L<T, D, 6>::run(a, st);
    case 7: return L<T, D, 7>::run(a, st);
    case 8: return L<T, D, 8>::run(a, st);
#endif
    default: return hipErrorInvalidValue;
  }
}
template <typename T, int D, int RBW>
struct LseLaunch {
  static hipError_t run(const CompressArgs& a, hipStream_t st) { return launch_lse_t<T, D, RBW>(a, st); }
};
template <typename T, int D, int RBW>
struct ColsumLaunch {
  static hipError_t run(const CompressArgs& a, hipStream_t st) { return launch_colsum_t<T, D, RBW>(a, st); }
};

template <typename T, int D>
static hipError_t launch_scores_d(const CompressArgs& a, hipStream_t st) {
  if (a.window_lse == nullptr) {
    const hipError_t e = dispatch_rbw<T, D, LseLaunch>(a.lse_rs_rows, a, st);
    if (e != hipSuccess) return e;
  }
  return dispatch_rbw<T, D, ColsumLaunch>(a.rs_rows, a, st);
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
