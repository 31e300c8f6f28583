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

// K tile staging: keys [tile0, tile0+64) of this head travel global -> registers
// (issued one tile ahead) -> LDS. Keys past the end of the head read as zeros.
template <typename T, int D>
struct KeyStage {
  using G = TileGeom<T, D>;
  static constexpr int N = (kScoreTile * G::V16) / kScoreBlock;  // 16-byte vectors per thread
  static_assert(N >= 1 && (kScoreTile * G::V16) % kScoreBlock == 0, "tile must split evenly");
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

// Pass 1: per-chunk partial log-sum-exp of every window row -------------------
//
// Each lane keeps, for each of its 4*RBW row slots, a reference m and a sum
// s = sum 2^(y - m) over the keys it has seen (y = logit*log2 e). m only
// moves when a value exceeds it by more than 64 (then the slot is updated
// exactly); otherwise s += 2^(y-m) costs one fma + one exp2 + one add.
// The sum stays below 2^64 * keys, far from fp32 overflow.
template <typename T, int D, int RBW>
__global__ __launch_bounds__(kScoreBlock, 1) void lse_kernel(CompressArgs a) {
  using G = TileGeom<T, D>;
  __shared__ __attribute__((aligned(16))) char ktile[kScoreTile * G::LDS_STRIDE];
  const int seg = blockIdx.y;
  const int b = seg / a.Hkv, h = seg % a.Hkv;
  const int64_t key0 = (int64_t)blockIdx.x * a.score_chunk;
  if (key0 >= a.C) return;
  const int64_t key_end = key0 + a.score_chunk < a.C ? key0 + a.score_chunk : a.C;
  const int tid = threadIdx.x, wid = tid >> 6, lane = tid & 63;
  const int lr = lane & 15, lg = lane >> 4;
  const int nrb = (a.R + 15) / 16;

  Frag<T> qa[RBW][G::NC];
  load_group_queries<T, D, RBW>(a, b, h, wid, lane, qa);
  const rsrc_t kr = make_rsrc(static_cast<const T*>(a.k) + (int64_t)seg * a.C * D,
                              (uint64_t)a.C * G::RB);

  // Causality: the row with window index i sees key j iff j - (C-w) <= i.
  // Rows past R see nothing.
  const int64_t vis0 = a.C - a.w;
  int wi[RBW][4];
  float m[RBW][4], s[RBW][4];
#pragma unroll
  for (int j = 0; j < RBW; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = (wid + kScoreWaves * j) * 16 + 4 * lg + i;
      wi[j][i] = row < a.R ? row % a.w : -(1 << 30);
      m[j][i] = -INFINITY;
      s[j][i] = 0.f;
    }
  const float c2 = a.c2;

  KeyStage<T, D> stage;
  stage.load(kr, key0);
  for (int64_t tile0 = key0; tile0 < key_end; tile0 += kScoreTile) {
    __syncthreads();
    stage.store(ktile);
    __syncthreads();
    if (tile0 + kScoreTile < key_end) stage.load(kr, tile0 + kScoreTile);
    const bool masked = tile0 + kScoreTile > vis0;  // uniform: tile reaches the window block
#pragma unroll 1
    for (int t = 0; t < kScoreTile / 16; ++t) {
      Frag<T> kb[G::NC];
#pragma unroll
      for (int c = 0; c < G::NC; ++c)
        kb[c] = lds_frag<T>(ktile, (uint32_t)((16 * t + lr) * G::LDS_STRIDE + (32 * c + 8 * lg) * G::EB));
      // key offset past the start of the window block, clamped into int range
      const int64_t dk64 = tile0 + 16 * t + lr - vis0;
      const int dk = dk64 < -(1 << 30) ? -(1 << 30) : (int)dk64;
      f32x4 acc[RBW];
      float tmax = -INFINITY;
#pragma unroll
      for (int j = 0; j < RBW; ++j) {
        if (wid + kScoreWaves * j < nrb) {
          acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int c = 0; c < G::NC; ++c) acc[j] = mma(qa[j][c], kb[c], acc[j]);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            float tv = fmaf(acc[j][i], c2, -m[j][i]);
            if (wi[j][i] < 0 || (masked && dk > wi[j][i])) tv = -INFINITY;  // padding / causal
            acc[j][i] = tv;
            tmax = fmaxf(tmax, tv);
          }
        } else {
          acc[j] = f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
        }
      }
      if (__any(tmax > 64.f)) {
        // Exact online update for this key: taken for the first key a slot sees
        // (m = -inf) and after jumps of more than 2^64. acc now holds t = y - m,
        // which is +inf while m is -inf, so the logits are recomputed.
#pragma unroll
        for (int j = 0; j < RBW; ++j) {
          if (wid + kScoreWaves * j >= nrb) continue;
          f32x4 z = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int c = 0; c < G::NC; ++c) z = mma(qa[j][c], kb[c], z);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const bool vis = !(masked && dk > wi[j][i]) && wi[j][i] >= 0;
            const float y = vis ? z[i] * c2 : -INFINITY;
            const float mn = fmaxf(m[j][i], y);
            if (mn != -INFINITY) {
              s[j][i] = s[j][i] * fast_exp2(m[j][i] - mn) + fast_exp2(y - mn);
              m[j][i] = mn;
            }
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < RBW; ++j)
#pragma unroll
          for (int i = 0; i < 4; ++i) s[j][i] += fast_exp2(acc[j][i]);
      }
    }
  }

  // Combine the 16 lanes (keys) of each row, then store (m, s) for the row.
  const int chunk = blockIdx.x;
  float* part = a.lse_part + ((int64_t)seg * a.n_lse_chunks + chunk) * a.R * 2;
  const rsrc_t pr = make_rsrc(part, (uint64_t)a.R * 2 * sizeof(float));
#pragma unroll
  for (int j = 0; j < RBW; ++j)
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

// Merge the per-chunk partials of every window row, in chunk order, in fp64.
__global__ __launch_bounds__(kBlock) void lse_merge_kernel(CompressArgs a) {
  const int64_t idx = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  const int64_t nrows = (int64_t)a.B * a.Hkv * a.R;
  if (idx >= nrows) return;
  const int64_t seg = idx / a.R, row = idx % a.R;
  const float* part = a.lse_part + (seg * a.n_lse_chunks) * a.R * 2;
  const rsrc_t pr = make_rsrc(part, (uint64_t)a.n_lse_chunks * a.R * 2 * sizeof(float));
  float mx = -INFINITY;
  for (int c = 0; c < a.n_lse_chunks; ++c)
    mx = fmaxf(mx, ldf(pr, (uint32_t)(((int64_t)c * a.R + row) * 8)));
  double sum = 0.0;
  if (mx != -INFINITY) {
    for (int c = 0; c < a.n_lse_chunks; ++c) {
      const float mc = ldf(pr, (uint32_t)(((int64_t)c * a.R + row) * 8));
      const float sc = ldf(pr, (uint32_t)(((int64_t)c * a.R + row) * 8 + 4));
      if (mc != -INFINITY) sum += (double)sc * exp2((double)mc - (double)mx);
    }
  }
  const float lse2 = (mx == -INFINITY || !(sum > 0.0)) ? -INFINITY : (float)((double)mx + log2(sum));
  const rsrc_t lr = make_rsrc(a.lse2, (uint64_t)nrows * sizeof(float));
  stf(lr, (uint32_t)(idx * 4), lse2);
}

// Pass 2: window-summed probabilities of every scored key --------------------
template <typename T, int D, int RBW>
__global__ __launch_bounds__(kScoreBlock, 1) void colsum_kernel(CompressArgs a) {
  using G = TileGeom<T, D>;
  __shared__ __attribute__((aligned(16))) char ktile[kScoreTile * G::LDS_STRIDE];
  __shared__ float red[kScoreWaves][kScoreTile];
  const int seg = blockIdx.y;
  const int b = seg / a.Hkv, h = seg % a.Hkv;
  const int64_t key0 = (int64_t)blockIdx.x * a.score_chunk;
  if (key0 >= a.n_scored) return;
  const int64_t key_end = key0 + a.score_chunk < a.n_scored ? key0 + a.score_chunk : a.n_scored;
  const int tid = threadIdx.x, wid = tid >> 6, lane = tid & 63;
  const int lr = lane & 15, lg = lane >> 4;
  const int nrb = (a.R + 15) / 16;

  Frag<T> qa[RBW][G::NC];
  load_group_queries<T, D, RBW>(a, b, h, wid, lane, qa);
  const rsrc_t kr = make_rsrc(static_cast<const T*>(a.k) + (int64_t)seg * a.C * D,
                              (uint64_t)a.C * G::RB);

  // -lse2 of this lane's row slots; rows past R get -inf so they add exp2(-inf) = 0
  const uint64_t nl = (uint64_t)a.B * a.Hkv * a.R;
  const bool natural = a.window_lse != nullptr;
  const rsrc_t lr2 = make_rsrc(natural ? (const void*)a.window_lse : (const void*)a.lse2,
                               nl * sizeof(float));
  float nlse[RBW][4];
#pragma unroll
  for (int j = 0; j < RBW; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = (wid + kScoreWaves * j) * 16 + 4 * lg + i;
      float l = ldf(lr2, (uint32_t)(((int64_t)seg * a.R + row) * 4));
      if (natural) l *= 1.44269504088896340736f;
      nlse[j][i] = row < a.R ? -l : -INFINITY;
    }
  const float c2 = a.c2;
  const rsrc_t cr = make_rsrc(a.colsum + (int64_t)seg * a.n_scored, (uint64_t)a.n_scored * 4);

  KeyStage<T, D> stage;
  stage.load(kr, key0);
  for (int64_t tile0 = key0; tile0 < key_end; tile0 += kScoreTile) {
    __syncthreads();
    stage.store(ktile);
    __syncthreads();
    if (tile0 + kScoreTile < key_end) stage.load(kr, tile0 + kScoreTile);
#pragma unroll 1
    for (int t = 0; t < kScoreTile / 16; ++t) {
      Frag<T> kb[G::NC];
#pragma unroll
      for (int c = 0; c < G::NC; ++c)
        kb[c] = lds_frag<T>(ktile, (uint32_t)((16 * t + lr) * G::LDS_STRIDE + (32 * c + 8 * lg) * G::EB));
      float p = 0.f;
#pragma unroll
      for (int j = 0; j < RBW; ++j) {
        if (wid + kScoreWaves * j < nrb) {
          f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int c = 0; c < G::NC; ++c) acc = mma(qa[j][c], kb[c], acc);
#pragma unroll
          for (int i = 0; i < 4; ++i) p += fast_exp2(fmaf(acc[i], c2, nlse[j][i]));
        }
      }
      p += __shfl_xor(p, 16, 64);
      p += __shfl_xor(p, 32, 64);
      if (lane < 16) red[wid][16 * t + lane] = p;
    }
    __syncthreads();
    if (tid < kScoreTile) {
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

// Host-side dispatch ----------------------------------------------------------
template <typename T, int D, int RBW>
static hipError_t launch_scores_t(const CompressArgs& a, hipStream_t st) {
  const dim3 sblk(kScoreBlock);
  if (a.window_lse == nullptr) {
    SGDKV_LAUNCH("score_lse", (lse_kernel<T, D, RBW>), dim3(a.n_lse_chunks, a.B * a.Hkv), sblk, st, a);
    const int64_t nrows = (int64_t)a.B * a.Hkv * a.R;
    SGDKV_LAUNCH("lse_merge", lse_merge_kernel, dim3((unsigned)((nrows + kBlock - 1) / kBlock)), dim3(kBlock), st, a);
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
