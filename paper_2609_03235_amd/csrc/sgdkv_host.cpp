// C ABI of the SGD-KV hot path: argument validation, head budget allocation
// (host), work planning and kernel launches. See include/sgdkv.h for the
// contract of every entry point.
//
// Compiled with -ffp-contract=off: the allocation's fp64 arithmetic decides
// integers, so every operation happens exactly in the order written.
#include "sgdkv.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <functional>
#include <mutex>
#include <queue>
#include <string>
#include <vector>

#include "sgdkv_internal.h"

namespace {

thread_local std::string g_error;

sgdkv_status fail(sgdkv_status code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_error = buf;
  return code;
}

sgdkv_status ok() {
  g_error.clear();
  return SGDKV_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
int64_t ceil_div(int64_t x, int64_t m) { return (x + m - 1) / m; }
size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// The kernels are built for gfx950 only; check the current device once per device.
// cus_out (optional) receives the device's compute-unit count.
sgdkv_status check_device(int* cus_out = nullptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(SGDKV_ERR_HIP, "no HIP device: %s", hipGetErrorString(e));
  static std::mutex mu;
  static std::vector<int> verdict;  // -1 unknown, 0 unsupported, 1 gfx950
  static std::vector<int> cus;
  std::lock_guard<std::mutex> lock(mu);
  if ((int)verdict.size() <= dev) {
    verdict.resize(dev + 1, -1);
    cus.resize(dev + 1, 0);
  }
  if (verdict[dev] < 0) {
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess) return fail(SGDKV_ERR_HIP, "hipGetDeviceProperties: %s", hipGetErrorString(e));
    verdict[dev] = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : 0;
    cus[dev] = prop.multiProcessorCount;
    if (!verdict[dev]) return fail(SGDKV_ERR_UNSUPPORTED, "device %d is %s; kernels are built for gfx950",
                                   dev, prop.gcnArchName);
  }
  if (!verdict[dev]) return fail(SGDKV_ERR_UNSUPPORTED, "device %d is not gfx950", dev);
  if (cus_out) *cus_out = cus[dev];
  return SGDKV_OK;
}

// ----------------------------------------------------------------- budgets
struct Ranked {
  double frac;
  double score;
  int64_t index;
};

// Largest-remainder rounding of real shares that sum to T. Ties: larger
// score, then lower index. Fp residue (never seen on well-posed inputs) is
// absorbed round-robin in the same order.
void round_shares(const std::vector<double>& x, const std::vector<double>& score, int64_t T,
                  std::vector<int64_t>& out) {
  const int64_t n = (int64_t)x.size();
  std::vector<Ranked> r(n);
  int64_t floors = 0, fractional = 0;
  for (int64_t h = 0; h < n; ++h) {
    const double f = std::floor(x[h]);
    out[h] = (int64_t)f;
    floors += out[h];
    r[h] = Ranked{x[h] - f, score[h], h};
    if (r[h].frac > 0.0) ++fractional;
  }
  std::sort(r.begin(), r.end(), [](const Ranked& a, const Ranked& b) {
    if (a.frac != b.frac) return a.frac > b.frac;
    if (a.score != b.score) return a.score > b.score;
    return a.index < b.index;
  });
  int64_t left = T - floors;
  const int64_t ones = left <= 0 ? 0 : std::min(left, fractional);
  for (int64_t k = 0; k < ones; ++k) out[r[k].index] += 1;
  left -= ones;
  for (int64_t k = 0; left > 0; k = (k + 1) % n, --left) out[r[k].index] += 1;
  for (int64_t k = 0; left < 0; k = (k + 1) % n) {
    const int64_t h = r[n - 1 - k].index;
    if (out[h] > 0) {
      out[h] -= 1;
      ++left;
    }
  }
}

// Heads in descending score order, ties to the lower index.
std::vector<int64_t> score_order(const std::vector<double>& score) {
  std::vector<int64_t> idx(score.size());
  for (size_t h = 0; h < idx.size(); ++h) idx[h] = (int64_t)h;
  std::sort(idx.begin(), idx.end(), [&](int64_t a, int64_t b) {
    if (score[a] != score[b]) return score[a] > score[b];
    return a < b;
  });
  return idx;
}

sgdkv_status check_sizes(int32_t L, int32_t H, int64_t C, int64_t s, int64_t W) {
  if (L < 1 || H < 1) return fail(SGDKV_ERR_INVALID_ARG, "L=%d and H=%d must be >= 1", L, H);
  if (C < 1) return fail(SGDKV_ERR_INVALID_ARG, "C=%lld must be >= 1", (long long)C);
  if (s < 0 || W < 0) return fail(SGDKV_ERR_INVALID_ARG, "b_sink and b_window must be >= 0");
  if (s + W > C) return fail(SGDKV_ERR_INVALID_ARG, "b_sink + b_window = %lld exceeds C = %lld",
                             (long long)(s + W), (long long)C);
  return SGDKV_OK;
}

}  // namespace

extern "C" {

const char* sgdkv_last_error(void) { return g_error.c_str(); }

int32_t sgdkv_version(void) { return 102; }

sgdkv_status sgdkv_reduce_query_head_scores(const double* per_qhead, int32_t L, int32_t Hq, int32_t Hkv,
                                            double* per_kvhead_out) {
  if (!per_qhead || !per_kvhead_out) return fail(SGDKV_ERR_INVALID_ARG, "NULL score pointer");
  if (L < 1 || Hq < 1 || Hkv < 1) return fail(SGDKV_ERR_INVALID_ARG, "L, Hq, Hkv must be >= 1");
  if (Hq % Hkv) return fail(SGDKV_ERR_INVALID_ARG, "Hq=%d is not a multiple of Hkv=%d", Hq, Hkv);
  const int32_t G = Hq / Hkv;
  for (int32_t l = 0; l < L; ++l)
    for (int32_t h = 0; h < Hkv; ++h) {
      const double* grp = per_qhead + (int64_t)l * Hq + (int64_t)h * G;
      per_kvhead_out[(int64_t)l * Hkv + h] = *std::max_element(grp, grp + G);
    }
  return ok();
}

sgdkv_status sgdkv_total_from_ratio(double R, int32_t L, int32_t H, int64_t C, int64_t b_sink,
                                    int64_t b_window, int32_t of_middle, int64_t* total_out) {
  if (!total_out) return fail(SGDKV_ERR_INVALID_ARG, "NULL total_out");
  if (!(R >= 0.0 && R <= 1.0)) return fail(SGDKV_ERR_INVALID_ARG, "ratio %g outside [0, 1]", R);
  if (sgdkv_status st = check_sizes(L, H, C, b_sink, b_window)) return st;
  const double LH = (double)L * (double)H;
  const int64_t reserved = (int64_t)L * H * (b_sink + b_window);
  int64_t total;
  if (of_middle) {
    total = reserved + (int64_t)std::floor(R * LH * (double)(C - b_sink - b_window));
  } else {
    total = (int64_t)std::floor(R * LH * (double)C);
    if (total < reserved)
      return fail(SGDKV_ERR_INVALID_ARG, "ratio %g gives %lld rows, fewer than the %lld sink+window rows",
                  R, (long long)total, (long long)reserved);
  }
  *total_out = total;
  return ok();
}

sgdkv_status sgdkv_allocate_budgets(const double* head_scores, int32_t L, int32_t H, int64_t C,
                                    int64_t b_sink, int64_t b_window, int64_t total_budget, int32_t mode,
                                    int64_t* budgets_out) {
  if (!head_scores || !budgets_out) return fail(SGDKV_ERR_INVALID_ARG, "NULL pointer");
  if (sgdkv_status st = check_sizes(L, H, C, b_sink, b_window)) return st;
  if (mode != 0 && mode != 1) return fail(SGDKV_ERR_INVALID_ARG, "mode %d is not 0 or 1", mode);
  const int64_t n = (int64_t)L * H;
  const int64_t reserve = b_sink + b_window;
  const int64_t M = C - reserve;
  if (total_budget < n * reserve || total_budget > n * C)
    return fail(SGDKV_ERR_INVALID_ARG, "total_budget %lld outside [%lld, %lld]", (long long)total_budget,
                (long long)(n * reserve), (long long)(n * C));
  double sum = 0.0;
  for (int64_t h = 0; h < n; ++h) {
    const double v = head_scores[h];
    if (!(v >= 0.0) || std::isinf(v)) return fail(SGDKV_ERR_INVALID_ARG, "score %lld is %g", (long long)h, v);
    sum += v;
  }
  if (std::isinf(sum)) return fail(SGDKV_ERR_INVALID_ARG, "scores sum to infinity");
  const int64_t T = total_budget - n * reserve;

  // Normalisation over all L*H heads (Sec. 3.3); all-zero scores mean uniform shares.
  std::vector<double> score(n);
  for (int64_t h = 0; h < n; ++h) score[h] = sum > 0.0 ? head_scores[h] : 1.0;
  const double denom = sum > 0.0 ? sum : (double)n;

  std::vector<double> share(n);
  std::vector<int64_t> mid(n);
  const std::vector<int64_t> order = score_order(score);
  if (mode == 0) {
    // Eq. 2 without the reserved rows (normalised score times T), rounded; then Algorithm 1.
    for (int64_t h = 0; h < n; ++h) share[h] = (score[h] / denom) * (double)T;
    round_shares(share, score, T, mid);
    int64_t excess = 0;
    for (int64_t h = 0; h < n; ++h)
      if (mid[h] > M) {
        excess += mid[h] - M;
        mid[h] = M;
      }
    for (int64_t h : order) {
      if (excess == 0) break;
      const int64_t give = std::min(M - mid[h], excess);
      if (give > 0) {
        mid[h] += give;
        excess -= give;
      }
    }
  } else {
    // Water level: share = min(lambda*score, M), summing to T. lambda*score is
    // evaluated as (score / uncapped score sum) * rows left, a fraction <= 1 of
    // the rows left, so tiny scores cannot overflow it.
    std::vector<double> tail(n + 1, 0.0);  // score sums over order[k..n-1], smallest first
    for (int64_t k = n - 1; k >= 0; --k) tail[k] = tail[k + 1] + score[order[k]];
    int64_t capped = 0;
    double left = (double)T, level = 0.0;
    bool flat = false;
    for (capped = 0; capped < n; ++capped) {
      left = (double)T - (double)capped * (double)M;
      if (tail[capped] <= 0.0) {
        flat = true;  // only zero-score heads remain: they share the rest evenly
        level = left / (double)(n - capped);
        break;
      }
      if ((score[order[capped]] / tail[capped]) * left <= (double)M) break;
    }
    for (int64_t k = 0; k < n; ++k) {
      const int64_t h = order[k];
      double v = k < capped ? (double)M : (flat ? level : (score[h] / tail[capped]) * left);
      share[h] = v > (double)M ? (double)M : v;
    }
    round_shares(share, score, T, mid);
    int64_t excess = 0;
    for (int64_t h = 0; h < n; ++h)
      if (mid[h] > M) {
        excess += mid[h] - M;
        mid[h] = M;
      }
    for (int64_t h : order) {
      if (excess == 0) break;
      const int64_t give = std::min(M - mid[h], excess);
      if (give > 0) {
        mid[h] += give;
        excess -= give;
      }
    }
  }
  for (int64_t h = 0; h < n; ++h) budgets_out[h] = reserve + mid[h];
  return ok();
}

sgdkv_status sgdkv_segment_offsets(const int64_t* layer_budgets, int32_t batch, int32_t num_kv_heads,
                                   int64_t* offsets_out) {
  if (!layer_budgets || !offsets_out) return fail(SGDKV_ERR_INVALID_ARG, "NULL pointer");
  if (batch < 1 || num_kv_heads < 1)
    return fail(SGDKV_ERR_INVALID_ARG, "batch=%d and num_kv_heads=%d must be >= 1", batch, num_kv_heads);
  const int64_t limit = (int64_t)1 << 62;
  int64_t T = 0;
  for (int32_t h = 0; h < num_kv_heads; ++h) {
    if (layer_budgets[h] < 0)
      return fail(SGDKV_ERR_INVALID_ARG, "layer_budgets[%d] = %lld < 0", h, (long long)layer_budgets[h]);
    if (layer_budgets[h] > limit / batch - T) return fail(SGDKV_ERR_INVALID_ARG, "batch * T_layer exceeds 2^62");
    T += layer_budgets[h];
  }
  for (int32_t b = 0; b < batch; ++b) {
    int64_t run = (int64_t)b * T;
    for (int32_t h = 0; h < num_kv_heads; ++h) {
      offsets_out[(int64_t)b * num_kv_heads + h] = run;
      run += layer_budgets[h];
    }
  }
  offsets_out[(int64_t)batch * num_kv_heads] = (int64_t)batch * T;
  return ok();
}

}  // extern "C"

// ------------------------------------------------------------ compress plan
namespace {

struct CompressPlan {
  sgdkv::CompressArgs a;
  size_t off_lse_part, off_lse2, off_colsum, off_pooled, off_hist, off_chunk_hist, bytes;
  int lse_chunks_max;  // pass-1 chunks any window position gives (sizes their partials)
  int colsum_splits;  // row splits the column-sum region has room for
};

// Row splits of a KV head's R = G*w window rows over score workgroups of at most kMaxSplitRows
// rows. Group mean and the weighted Ipt. modes: as even as whole 16-row blocks allow. Ipt. max:
// whole query heads per split (w % 16 == 0 and w <= kMaxSplitRows, checked by the caller).
void row_splits(int R, int w, bool whole_heads, int& n, int& rows) {
  if (whole_heads) {
    const int heads = sgdkv::kMaxSplitRows / w;
    rows = heads * w;
    n = (int)ceil_div(R, rows);
  } else {
    n = (int)ceil_div(R, sgdkv::kMaxSplitRows);
    rows = (int)round_up(ceil_div(R, n), 16);
  }
  if (n == 1) rows = R;
}

// win0 = position of the first window row (seq_len - obs_window for the default window); the
// workspace is sized for any win0 (scores for up to seq_len keys), so its size depends on d only.
sgdkv_status plan_compress(const sgdkv_compress_desc* d, int64_t win0, CompressPlan& p) {
  if (!d) return fail(SGDKV_ERR_INVALID_ARG, "NULL descriptor");
  if (d->batch < 1 || d->num_q_heads < 1 || d->num_kv_heads < 1)
    return fail(SGDKV_ERR_INVALID_ARG, "batch, num_q_heads, num_kv_heads must be >= 1");
  if (d->num_q_heads % d->num_kv_heads)
    return fail(SGDKV_ERR_INVALID_ARG, "num_q_heads %d is not a multiple of num_kv_heads %d", d->num_q_heads,
                d->num_kv_heads);
  if (d->num_kv_heads > sgdkv::kMaxKvHeads)
    return fail(SGDKV_ERR_UNSUPPORTED, "num_kv_heads %d > %d", d->num_kv_heads, sgdkv::kMaxKvHeads);
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(SGDKV_ERR_UNSUPPORTED, "head_dim %d (built: 64, 128)", d->head_dim);
  if (d->dtype != SGDKV_DTYPE_F32 && d->dtype != SGDKV_DTYPE_BF16)
    return fail(SGDKV_ERR_INVALID_ARG, "dtype %d", d->dtype);
  if (d->obs_window < 1) return fail(SGDKV_ERR_INVALID_ARG, "obs_window must be >= 1");
  if (d->pool_kernel < 1 || d->pool_kernel % 2 == 0)
    return fail(SGDKV_ERR_INVALID_ARG, "pool_kernel %d must be odd and >= 1", d->pool_kernel);
  if (d->seq_len < 1 || d->seq_len > 0x7FFFFFFFll)
    return fail(SGDKV_ERR_INVALID_ARG, "seq_len %lld outside [1, 2^31-1]", (long long)d->seq_len);
  if (d->b_sink < 0 || d->b_window < 0) return fail(SGDKV_ERR_INVALID_ARG, "b_sink, b_window must be >= 0");
  if (d->b_sink + d->b_window > d->seq_len) return fail(SGDKV_ERR_INVALID_ARG, "b_sink + b_window > seq_len");
  if (win0 < 0 || win0 > d->seq_len)
    return fail(SGDKV_ERR_INVALID_ARG, "window position %lld outside [0, seq_len]", (long long)win0);
  if (d->b_window < d->seq_len - win0)
    return fail(SGDKV_ERR_INVALID_ARG,
                "b_window %lld < %lld (keys from the window on): recent candidates would have no score",
                (long long)d->b_window, (long long)(d->seq_len - win0));
  if (!(d->scale >= 0.f) || std::isinf(d->scale)) return fail(SGDKV_ERR_INVALID_ARG, "scale %g", d->scale);
  const int G = d->num_q_heads / d->num_kv_heads;
  const int64_t R = (int64_t)G * d->obs_window;
  if (R > sgdkv::kMaxGroupRows)
    return fail(SGDKV_ERR_UNSUPPORTED, "group rows G*w = %lld > %d", (long long)R, sgdkv::kMaxGroupRows);
  if ((int64_t)d->batch * d->num_kv_heads > 65535)
    return fail(SGDKV_ERR_UNSUPPORTED, "batch * num_kv_heads = %lld > 65535",
                (long long)d->batch * d->num_kv_heads);
  const int eb = d->dtype == SGDKV_DTYPE_BF16 ? 2 : 4;
  const int64_t rb = (int64_t)d->head_dim * eb;
  // kernels address one head's keys, plus a margin of 256 key rows read past its end, in 32 bits
  if ((d->seq_len + 256) * rb > 0xFFFFFFFFll)
    return fail(SGDKV_ERR_UNSUPPORTED, "one head's keys (%lld bytes) exceed 4 GiB less 256 rows",
                (long long)(d->seq_len * rb));

  sgdkv::CompressArgs& a = p.a;
  std::memset(&a, 0, sizeof a);
  a.B = d->batch;
  a.Hq = d->num_q_heads;
  a.Hkv = d->num_kv_heads;
  a.G = G;
  a.D = d->head_dim;
  a.w = d->obs_window;
  a.kp = d->pool_kernel;
  a.R = (int)R;
  a.dtype = d->dtype;
  a.C = d->seq_len;
  a.s = d->b_sink;
  a.W = d->b_window;
  a.win0 = win0;
  a.n_scored = win0;
  const double scale = d->scale > 0.f ? (double)d->scale : 1.0 / std::sqrt((double)d->head_dim);
  a.c2 = (float)(scale * 1.4426950408889634074);
  a.out_scale = 1.0f / (float)G;
  row_splits(a.R, a.w, false, a.n_rsplit, a.rs_rows);
  a.lse_n_rsplit = a.n_rsplit;  // pass 1 keeps the even split (Ipt. max changes pass 2's only)
  a.lse_rs_rows = a.rs_rows;
  // the column-sum region also fits the (possibly more) splits of the Ipt. max aggregation
  p.colsum_splits = a.n_rsplit;
  if (a.w % 16 == 0 && a.w <= sgdkv::kMaxSplitRows) {
    int n_heads_split = 0, rows = 0;
    row_splits(a.R, a.w, true, n_heads_split, rows);
    p.colsum_splits = std::max(p.colsum_splits, n_heads_split);
  }

  const int64_t nseg = (int64_t)a.B * a.Hkv;
  // score workgroups: about one per compute unit in total (one round of one resident workgroup per
  // CU: fewer, longer workgroups measured faster than two rounds, and 1.5 rounds leave the second
  // half empty), counting each row split; a chunk is a whole number of key tiles, so no tile of
  // pass 1 reaches into the next chunk (which would count those keys twice). The chunk does not
  // depend on the aggregation, so neither does the workspace.
  a.score_chunk = std::min<int64_t>(
      std::max<int64_t>(round_up(ceil_div(nseg * a.n_rsplit * a.C, sgdkv::kScoreWorkgroups), sgdkv::kScoreChunkQuantum),
                        2 * sgdkv::kScoreChunkQuantum),
      1 << 16);
  // pass 1 covers the keys some window row sees, [0, min(C, win0 + w)), in uniform chunks (about
  // one workgroup per CU). The chunk holding the causally masked tiles runs them on the exact
  // path, which then ends the launch. Where that costs more than what splitting those tiles off
  // into a short chunk of their own costs -- its workgroups (one per segment and row split, on
  // the exact path, dispatched first) leave their CUs idle for the rest of the launch, about
  // tiles-per-chunk x tails / (256 CUs) tile times, against about two for the exact tiles --
  // the masked tiles get that chunk, and the uniform chunks aim at the CUs the tails leave. The
  // chunk sizes depend on C only, so the workspace does not depend on win0.
  {
    const int64_t tails = nseg * a.n_rsplit;
    const int64_t vis_end = std::min<int64_t>(a.C, win0 + a.w);
    const int64_t open_end = std::min<int64_t>(a.C, win0);
    auto chunk_for = [&](int64_t target) {
      return std::min<int64_t>(
          std::max<int64_t>(round_up(ceil_div(tails * a.C, target), sgdkv::kScoreChunkQuantum),
                            2 * sgdkv::kScoreChunkQuantum),
          1 << 16);
    };
    a.lse_chunk = chunk_for(sgdkv::kScoreWorkgroups);
    const bool split_tail = (a.lse_chunk / sgdkv::kLseTile) * tails < 2 * sgdkv::kScoreWorkgroups &&
                            tails < sgdkv::kScoreWorkgroups;
    if (split_tail) {
      a.lse_chunk = chunk_for(sgdkv::kScoreWorkgroups - tails);
      a.lse_tail0 = open_end / sgdkv::kLseTile * sgdkv::kLseTile;
    } else {
      a.lse_tail0 = vis_end;  // no tail chunk: the last uniform chunk holds the masked tiles
    }
    a.n_lse_head = (int)ceil_div(a.lse_tail0, a.lse_chunk);
    a.n_lse_chunks = a.n_lse_head + (vis_end > a.lse_tail0 ? 1 : 0);
    p.lse_chunks_max = (int)ceil_div(a.C, a.lse_chunk) + 1;
  }
  a.n_col_chunks = (int)ceil_div(a.n_scored, a.score_chunk);
  // pooling, radix and compaction passes: about 1024 workgroups, of 1024 to kHistChunkMax positions
  // (fewer, longer chunks at small sizes: the compaction adds up the chunks before its own)
  a.hist_chunk = std::min<int64_t>(std::max<int64_t>(round_up(ceil_div(nseg * a.n_scored, 1024), 256), 1024),
                                   sgdkv::kHistChunkMax);
  a.n_hist_chunks = (int)ceil_div(a.n_scored, a.hist_chunk);
  a.n_cmp_chunks = (int)ceil_div(a.C, a.hist_chunk);

  size_t off = 0;
  p.off_lse_part = off;
  off += align256((size_t)nseg * p.lse_chunks_max * R * 2 * sizeof(float));
  p.off_lse2 = off;
  off += align256((size_t)nseg * R * sizeof(float));
  p.off_colsum = off;
  off += align256((size_t)p.colsum_splits * nseg * a.C * sizeof(float));
  p.off_pooled = off;
  off += align256((size_t)nseg * a.C * sizeof(float));
  p.off_hist = off;
  off += align256((size_t)nseg * 4 * 256 * sizeof(uint32_t));  // one 256-bin histogram per radix digit
  p.off_chunk_hist = off;
  off += align256((size_t)nseg * a.n_hist_chunks * sgdkv::kChunkHistWords * sizeof(uint32_t));
  p.bytes = off;
  return SGDKV_OK;
}

}  // namespace

extern "C" {

sgdkv_status sgdkv_allocate_budgets_variant(const double* head_scores, const double* second_scores, int32_t L,
                                            int32_t H, int64_t C, int64_t b_sink, int64_t b_window,
                                            int64_t total_budget, int32_t mode, int32_t variant,
                                            double full_fraction, int64_t* budgets_out) {
  if (!head_scores || !budgets_out) return fail(SGDKV_ERR_INVALID_ARG, "NULL pointer");
  if (sgdkv_status st = check_sizes(L, H, C, b_sink, b_window)) return st;
  const int64_t n = (int64_t)L * H;
  const int64_t reserve = b_sink + b_window;
  const int64_t M = C - reserve;
  for (int64_t h = 0; h < n; ++h)
    if (!(head_scores[h] >= 0.0) || std::isinf(head_scores[h]))
      return fail(SGDKV_ERR_INVALID_ARG, "score %lld is %g", (long long)h, head_scores[h]);
  switch (variant) {
    case SGDKV_ALLOC_PLAIN:
      return sgdkv_allocate_budgets(head_scores, L, H, C, b_sink, b_window, total_budget, mode, budgets_out);
    case SGDKV_ALLOC_THR: {
      double sum = 0.0;
      for (int64_t h = 0; h < n; ++h) sum += head_scores[h];
      const double mean = sum / (double)n;
      std::vector<double> kept(n);
      for (int64_t h = 0; h < n; ++h) kept[h] = head_scores[h] < mean ? 0.0 : head_scores[h];
      return sgdkv_allocate_budgets(kept.data(), L, H, C, b_sink, b_window, total_budget, mode, budgets_out);
    }
    case SGDKV_ALLOC_REVERSE: {
      std::vector<int64_t> plain(n);
      if (sgdkv_status st =
              sgdkv_allocate_budgets(head_scores, L, H, C, b_sink, b_window, total_budget, mode, plain.data()))
        return st;
      for (int64_t h = 0; h < n; ++h) budgets_out[h] = reserve + (M - (plain[h] - reserve));
      return ok();
    }
    case SGDKV_ALLOC_MIX: {
      if (!second_scores) return fail(SGDKV_ERR_INVALID_ARG, "the mix variant needs second_scores");
      double s1 = 0.0, s2 = 0.0;
      for (int64_t h = 0; h < n; ++h) {
        if (!(second_scores[h] >= 0.0) || std::isinf(second_scores[h]))
          return fail(SGDKV_ERR_INVALID_ARG, "second score %lld is %g", (long long)h, second_scores[h]);
        s1 += head_scores[h];
        s2 += second_scores[h];
      }
      if (std::isinf(s1) || std::isinf(s2)) return fail(SGDKV_ERR_INVALID_ARG, "scores sum to infinity");
      std::vector<double> avg(n);
      for (int64_t h = 0; h < n; ++h) {
        const double u = s1 > 0.0 ? head_scores[h] / s1 : 1.0 / (double)n;
        const double v = s2 > 0.0 ? second_scores[h] / s2 : 1.0 / (double)n;
        avg[h] = (u + v) / 2.0;
      }
      return sgdkv_allocate_budgets(avg.data(), L, H, C, b_sink, b_window, total_budget, mode, budgets_out);
    }
    case SGDKV_ALLOC_BINARY:
    case SGDKV_ALLOC_BINARY_REVERSE: {
      if (!(full_fraction >= 0.0 && full_fraction <= 1.0))
        return fail(SGDKV_ERR_INVALID_ARG, "full_fraction %g outside [0, 1]", full_fraction);
      const int64_t k = (int64_t)std::floor(full_fraction * (double)n);
      const std::vector<int64_t> order = score_order(std::vector<double>(head_scores, head_scores + n));
      for (int64_t h = 0; h < n; ++h) budgets_out[h] = reserve;
      for (int64_t j = 0; j < k; ++j) budgets_out[order[variant == SGDKV_ALLOC_BINARY ? j : n - 1 - j]] = C;
      return ok();
    }
    default:
      return fail(SGDKV_ERR_INVALID_ARG, "unknown allocation variant %d", variant);
  }
}

sgdkv_status sgdkv_compress_workspace_size(const sgdkv_compress_desc* desc, size_t* bytes) {
  if (!bytes) return fail(SGDKV_ERR_INVALID_ARG, "NULL bytes");
  if (!desc) return fail(SGDKV_ERR_INVALID_ARG, "NULL descriptor");
  CompressPlan p;
  // the size does not depend on the window position; plan with the one every b_window allows
  if (sgdkv_status st = plan_compress(desc, desc->seq_len, p)) return st;
  *bytes = p.bytes;
  return ok();
}

sgdkv_status sgdkv_compress_layer(const sgdkv_compress_desc* desc, const int64_t* layer_budgets,
                                  const void* q_win, const void* k, const void* v, const float* window_lse,
                                  void* k_out, void* v_out, int32_t* kept_pos_out, int64_t* offsets_out,
                                  float* scores_out, void* workspace, size_t workspace_bytes, void* stream) {
  return sgdkv_compress_layer_ex(desc, nullptr, layer_budgets, q_win, k, v, window_lse, k_out, v_out,
                                 kept_pos_out, offsets_out, scores_out, workspace, workspace_bytes, stream);
}

sgdkv_status sgdkv_compress_layer_ex(const sgdkv_compress_desc* desc, const sgdkv_compress_opts* opts,
                                     const int64_t* layer_budgets, const void* q_win, const void* k,
                                     const void* v, const float* window_lse, void* k_out, void* v_out,
                                     int32_t* kept_pos_out, int64_t* offsets_out, float* scores_out,
                                     void* workspace, size_t workspace_bytes, void* stream) {
  sgdkv_compress_opts o{SGDKV_GROUP_MEAN, 0, nullptr, -1, nullptr};
  if (opts) o = *opts;
  if (!desc) return fail(SGDKV_ERR_INVALID_ARG, "NULL descriptor");
  if (o.reserved != 0) return fail(SGDKV_ERR_INVALID_ARG, "opts.reserved must be 0");
  if (o.window_pos < -1) return fail(SGDKV_ERR_INVALID_ARG, "window_pos %lld < -1", (long long)o.window_pos);
  const int64_t win0 = o.window_pos == -1 ? desc->seq_len - desc->obs_window : o.window_pos;
  CompressPlan p;
  if (sgdkv_status st = plan_compress(desc, win0, p)) return st;
  sgdkv::CompressArgs& a = p.a;
  const int32_t group_agg = o.group_agg;
  const double* qhead_scores = o.qhead_scores;
  if (group_agg < SGDKV_GROUP_MEAN || group_agg > SGDKV_GROUP_IPT_ONLY)
    return fail(SGDKV_ERR_INVALID_ARG, "group_agg %d is not 0..3", group_agg);
  a.agg = group_agg;
  if (group_agg != SGDKV_GROUP_MEAN) {
    if (!qhead_scores) return fail(SGDKV_ERR_INVALID_ARG, "group_agg %d needs qhead_scores", group_agg);
    if (a.Hq > sgdkv::kMaxIptQHeads)
      return fail(SGDKV_ERR_UNSUPPORTED, "num_q_heads %d > %d with an Ipt. aggregation", a.Hq, sgdkv::kMaxIptQHeads);
    if (group_agg == SGDKV_GROUP_IPT_MAX && (a.w % 16 != 0 || a.w > sgdkv::kMaxSplitRows))
      return fail(SGDKV_ERR_UNSUPPORTED, "Ipt. max needs obs_window %% 16 == 0 and <= %d (got %d)",
                  sgdkv::kMaxSplitRows, a.w);
    if (group_agg == SGDKV_GROUP_IPT_MAX) row_splits(a.R, a.w, true, a.n_rsplit, a.rs_rows);
    for (int q = 0; q < a.Hq; ++q)
      if (!(qhead_scores[q] >= 0.0) || std::isinf(qhead_scores[q]))
        return fail(SGDKV_ERR_INVALID_ARG, "qhead_scores[%d] is %g", q, qhead_scores[q]);
    for (int h = 0; h < a.Hkv; ++h) {
      int top = 0;  // the group's highest score, lower query head on ties
      for (int g = 1; g < a.G; ++g)
        if (qhead_scores[h * a.G + g] > qhead_scores[h * a.G + top]) top = g;
      for (int g = 0; g < a.G; ++g) {
        const double sc = qhead_scores[h * a.G + g];
        float wgt;
        if (group_agg == SGDKV_GROUP_IPT_MAX) wgt = (float)sc;
        else if (group_agg == SGDKV_GROUP_IPT_MEAN) wgt = sc > 0.0 ? (float)std::log2(sc) : -INFINITY;
        else wgt = g == top ? 0.0f : -INFINITY;
        a.qweight[h * a.G + g] = wgt;
      }
    }
    a.out_scale = group_agg == SGDKV_GROUP_IPT_MEAN ? 1.0f / (float)a.G : 1.0f;
  }
  const int n_out = (k_out != nullptr) + (v_out != nullptr) + (kept_pos_out != nullptr) + (offsets_out != nullptr);
  if (n_out != 0 && n_out != 4)
    return fail(SGDKV_ERR_INVALID_ARG, "k_out, v_out, kept_pos_out, offsets_out must be all set or all NULL");
  const bool scores_only = n_out == 0;
  if (scores_only && !scores_out) return fail(SGDKV_ERR_INVALID_ARG, "scores-only mode needs scores_out");
  if (!q_win || !k) return fail(SGDKV_ERR_INVALID_ARG, "NULL q_win or k");
  if (!scores_only && !v) return fail(SGDKV_ERR_INVALID_ARG, "NULL v");
  const void* ptrs[] = {q_win, k, v, window_lse, k_out, v_out, kept_pos_out, offsets_out, scores_out};
  const char* names[] = {"q_win", "k", "v", "window_lse", "k_out", "v_out", "kept_pos_out", "offsets_out",
                         "scores_out"};
  for (int i = 0; i < 9; ++i)
    if (ptrs[i] && !aligned16(ptrs[i])) return fail(SGDKV_ERR_INVALID_ARG, "%s is not 16-byte aligned", names[i]);
  if (!scores_only || layer_budgets) {
    if (!layer_budgets) return fail(SGDKV_ERR_INVALID_ARG, "NULL layer_budgets");
    int64_t run = 0;
    for (int h = 0; h < a.Hkv; ++h) {
      const int64_t bh = layer_budgets[h];
      if (bh < a.s + a.W || bh > a.C)
        return fail(SGDKV_ERR_INVALID_ARG, "layer_budgets[%d] = %lld outside [%lld, %lld]", h, (long long)bh,
                    (long long)(a.s + a.W), (long long)a.C);
      a.m[h] = bh - a.s - a.W;
      a.prefix[h] = run;
      run += bh;
    }
    a.prefix[a.Hkv] = run;
    a.T_layer = run;
    int64_t longest = 0;
    for (int h = 0; h < a.Hkv; ++h) longest = std::max<int64_t>(longest, layer_budgets[h]);
    a.copy_blocks = scores_only ? 0 : (int)ceil_div(longest, sgdkv::kCopyRows);
  }
  if (p.bytes > 0) {
    if (!workspace) return fail(SGDKV_ERR_WORKSPACE, "NULL workspace (%zu bytes needed)", p.bytes);
    if (reinterpret_cast<uintptr_t>(workspace) & 255u)
      return fail(SGDKV_ERR_WORKSPACE, "workspace is not 256-byte aligned");
    if (workspace_bytes < p.bytes)
      return fail(SGDKV_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", workspace_bytes, p.bytes);
  }
  int cus = 0;
  if (sgdkv_status st = check_device(&cus)) return st;

  char* ws = static_cast<char*>(workspace);
  a.q_win = q_win;
  a.k = k;
  a.v = v;
  a.window_lse = window_lse;
  a.k_out = k_out;
  a.v_out = v_out;
  a.kept_pos = kept_pos_out;
  a.offsets = offsets_out;
  a.pooled = scores_out ? scores_out : reinterpret_cast<float*>(ws + p.off_pooled);
  a.lse_part = reinterpret_cast<float*>(ws + p.off_lse_part);
  a.lse2 = reinterpret_cast<float*>(ws + p.off_lse2);
  a.colsum = reinterpret_cast<float*>(ws + p.off_colsum);
  a.hist = reinterpret_cast<uint32_t*>(ws + p.off_hist);
  a.chunk_hist = reinterpret_cast<uint32_t*>(ws + p.off_chunk_hist);

  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = hipGetLastError();  // clear a stale error left by earlier, unrelated work
  (void)e;
  // With a gather stream, the gather waits for the selection through an event, then runs on
  // its own stream with half as many workgroups as the device has compute units, so that it
  // fits beside whatever the caller enqueues next on `stream`. The event is created before
  // anything is enqueued.
  hipStream_t gs = static_cast<hipStream_t>(o.gather_stream);
  const bool side = !scores_only && gs && gs != st;
  hipEvent_t ev = nullptr;
  if (side) {
    e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
    if (e != hipSuccess) return fail(SGDKV_ERR_HIP, "hipEventCreateWithFlags: %s", hipGetErrorString(e));
  }
  auto release = [&]() {
    if (ev) (void)hipEventDestroy(ev);  // released once the recorded work completes
  };
  e = sgdkv::launch_scores(a, st);
  if (e == hipSuccess) e = sgdkv::launch_select(a, scores_only, st);
  if (e != hipSuccess) {
    release();
    return fail(SGDKV_ERR_HIP, "score or selection kernels: %s", hipGetErrorString(e));
  }
  if (scores_only) return ok();
  if (side) {
    e = hipEventRecord(ev, st);
    if (e == hipSuccess) e = hipStreamWaitEvent(gs, ev, 0);
    release();
    if (e == hipSuccess) e = sgdkv::launch_gather(a, std::max(1, cus / 2), gs);
  } else {
    e = sgdkv::launch_gather(a, 0, st);
  }
  if (e != hipSuccess) return fail(SGDKV_ERR_HIP, "gather: %s", hipGetErrorString(e));
  return ok();
}

}  // extern "C"

// -------------------------------------------------------------- decode plan
namespace {

#ifndef SGDKV_DECODE_SPLITS
#define SGDKV_DECODE_SPLITS 12288
#endif
#ifndef SGDKV_DECODE_MIN_CHUNK
#define SGDKV_DECODE_MIN_CHUNK 128
#endif
#ifndef SGDKV_DECODE_WHOLE_ROUNDS
#define SGDKV_DECODE_WHOLE_ROUNDS 1
#endif
constexpr int64_t kDecodeSplits = SGDKV_DECODE_SPLITS;
constexpr int64_t kDecodeMinChunk = SGDKV_DECODE_MIN_CHUNK;
constexpr bool kDecodeWholeRounds = SGDKV_DECODE_WHOLE_ROUNDS != 0;
// decode workgroups the MI355X runs at once: two per compute unit (their registers), 256 units
constexpr int64_t kDecodeResident = 2 * sgdkv::kScoreWorkgroups;

// Workgroups of each segment's compressed rows on the compact grid. Each workgroup's four waves
// are four splits of about chunk rows, which gives w0 workgroups in all. The device runs
// kDecodeResident of them at once and starts the next one where one ends, so a grid of, say,
// 3.7 rounds leaves a quarter of the device idle for a workgroup's length at its end. With more
// than one round, the workgroups are therefore shared out over the segments in proportion to
// their 16-row steps (largest remainder, ties to the lower segment; a non-empty segment left
// with none gets one from the largest) so that they fill a whole number of rounds, the one at or
// below w0 (fewer, longer workgroups: at a 10 % budget of 128K x B 8, 1.6 rounds became one, not
// two, 3 % faster; the larger caches measured alike); the kernel deals a segment's steps to four
// splits per launched workgroup. The new_wg workgroups of
// each segment's appended rows count toward the rounds when they come to at most half a round, so
// that they fill the last one instead of starting another.
std::vector<int64_t> compact_workgroups(const int64_t* offsets_host, int64_t nseg, int64_t chunk,
                                        int64_t new_wg = 0) {
  const int64_t wpw = sgdkv::kDecodeWaves;
  std::vector<int64_t> n((size_t)nseg);
  int64_t w0 = 0, steps = 0;
  for (int64_t i = 0; i < nseg; ++i) {
    const int64_t len = offsets_host[i + 1] - offsets_host[i];
    n[i] = ceil_div(ceil_div(len, chunk), wpw);
    w0 += n[i];
    steps += ceil_div(len, 16);
  }
  if (!kDecodeWholeRounds || w0 <= kDecodeResident) return n;
  const int64_t extra = nseg * new_wg <= kDecodeResident / 2 ? nseg * new_wg : 0;
  const int64_t target = (w0 + extra) / kDecodeResident * kDecodeResident - extra;
  std::vector<std::pair<int64_t, int64_t>> rem;  // (fractional part scaled by steps, -segment)
  int64_t given = 0;
  for (int64_t i = 0; i < nseg; ++i) {
    const int64_t st = ceil_div(offsets_host[i + 1] - offsets_host[i], 16);
    n[i] = target * st / steps;
    rem.emplace_back(target * st % steps, -i);
    given += n[i];
  }
  std::sort(rem.begin(), rem.end(), std::greater<>());
  for (int64_t j = 0; j < target - given; ++j) n[(size_t)-rem[(size_t)j].second] += 1;
  // a non-empty segment whose share rounded to none gets one, taken from the largest segment
  // (ties: the lower one)
  std::priority_queue<std::pair<int64_t, int64_t>> big;  // (workgroups, -segment)
  for (int64_t i = 0; i < nseg; ++i) big.emplace(n[i], -i);
  for (int64_t i = 0; i < nseg; ++i) {
    if (n[i] != 0 || offsets_host[i + 1] == offsets_host[i]) continue;
    n[i] = 1;
    const int64_t b = -big.top().second;
    big.pop();
    if (n[b] > 1) n[b] -= 1;
    big.emplace(n[b], -b);
  }
  return n;
}

struct DecodePlan {
  sgdkv::DecodeArgs a;
  size_t bytes;
};

sgdkv_status plan_decode(const sgdkv_decode_desc* d, const int64_t* offsets_host, int64_t capacity, DecodePlan& p) {
  if (!d) return fail(SGDKV_ERR_INVALID_ARG, "NULL descriptor");
  if (capacity < 0) return fail(SGDKV_ERR_INVALID_ARG, "capacity %lld < 0", (long long)capacity);
  if (!offsets_host) return fail(SGDKV_ERR_INVALID_ARG, "NULL offsets_host");
  if (d->batch < 1 || d->num_q_heads < 1 || d->num_kv_heads < 1)
    return fail(SGDKV_ERR_INVALID_ARG, "batch, num_q_heads, num_kv_heads must be >= 1");
  if (d->num_q_heads % d->num_kv_heads)
    return fail(SGDKV_ERR_INVALID_ARG, "num_q_heads %d is not a multiple of num_kv_heads %d", d->num_q_heads,
                d->num_kv_heads);
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(SGDKV_ERR_UNSUPPORTED, "head_dim %d (built: 64, 128)", d->head_dim);
  if ((d->kv_dtype != 0 && d->kv_dtype != 1) || (d->out_dtype != 0 && d->out_dtype != 1))
    return fail(SGDKV_ERR_INVALID_ARG, "dtype");
  const int G = d->num_q_heads / d->num_kv_heads;
  if (G > sgdkv::kMaxDecodeGroup) return fail(SGDKV_ERR_UNSUPPORTED, "group size %d > %d", G, sgdkv::kMaxDecodeGroup);
  if (!(d->scale >= 0.f) || std::isinf(d->scale)) return fail(SGDKV_ERR_INVALID_ARG, "scale %g", d->scale);
  const int64_t nseg = (int64_t)d->batch * d->num_kv_heads;
  if (nseg > 65535) return fail(SGDKV_ERR_UNSUPPORTED, "batch * num_kv_heads = %lld > 65535", (long long)nseg);
  if ((int64_t)d->batch * d->num_q_heads > 0x7FFFFFFFll) return fail(SGDKV_ERR_UNSUPPORTED, "batch * num_q_heads");
  const int64_t rb = (int64_t)d->head_dim * (d->kv_dtype == 1 ? 2 : 4);
  if (offsets_host[0] < 0) return fail(SGDKV_ERR_INVALID_ARG, "offsets[0] < 0");
  int64_t longest = 0;
  for (int64_t i = 0; i < nseg; ++i) {
    const int64_t len = offsets_host[i + 1] - offsets_host[i];
    if (len < 0) return fail(SGDKV_ERR_INVALID_ARG, "offsets decrease at %lld", (long long)i);
    longest = std::max(longest, len);
  }
  if (longest * rb > 0xFFFFFFFFll) return fail(SGDKV_ERR_UNSUPPORTED, "a segment exceeds 4 GiB");
  const int64_t total = offsets_host[nseg];

  sgdkv::DecodeArgs& a = p.a;
  std::memset(&a, 0, sizeof a);
  a.B = d->batch;
  a.Hq = d->num_q_heads;
  a.Hkv = d->num_kv_heads;
  a.G = G;
  a.D = d->head_dim;
  a.kv_dtype = d->kv_dtype;
  a.out_dtype = d->out_dtype;
  const double scale = d->scale > 0.f ? (double)d->scale : 1.0 / std::sqrt((double)d->head_dim);
  a.c2 = (float)(scale * 1.4426950408889634074);
  a.total_rows = total;
  // rows per wave-sized split: about kDecodeSplits splits over the whole batch, at least
  // kDecodeMinChunk rows; one round of longer splits measured slower
  a.chunk = std::min<int64_t>(
      std::max<int64_t>(round_up(ceil_div(total - offsets_host[0], kDecodeSplits), 64), kDecodeMinChunk), 1 << 24);
  // a batch whose minimum-size splits would launch fewer workgroups than the device has compute
  // units gets splits half as long (64 rows measured best at 32K x B 1: shorter ones add more
  // partials to combine than they save); one that would launch more than two rounds of them gets
  // splits twice as long (fewer workgroups, each with less of its fixed cost per row, and fewer
  // partials to combine: decode per 128K x B 8 layer -3.7 %; the 256K x B 16 and 1M x B 32 caches
  // already have splits of 512 rows and more)
  const int wpw = sgdkv::kDecodeWaves;  // splits (waves) per decode workgroup
  if (a.chunk == kDecodeMinChunk) {
    int64_t wgs = 0;
    for (int64_t i = 0; i < nseg; ++i) wgs += ceil_div(ceil_div(offsets_host[i + 1] - offsets_host[i], a.chunk), wpw);
    if (wgs < sgdkv::kScoreWorkgroups) a.chunk = kDecodeMinChunk / 2;
    else if (wgs > 2 * kDecodeResident) a.chunk = kDecodeMinChunk * 2;
  }
  a.n_chunk_max = (int)ceil_div(longest, a.chunk);
  if ((int64_t)a.B * a.Hkv * capacity * rb > 0xFFFFFFFFll)
    return fail(SGDKV_ERR_UNSUPPORTED, "appended regions of %lld rows per head exceed 4 GiB", (long long)capacity);
  a.cap = capacity;
  a.n_cwg = (int)ceil_div(a.n_chunk_max, wpw);
  // one partial slot per launched workgroup: with the compact grid each segment's own
  // workgroups (so the workspace follows the total of the splits, not the longest segment),
  // otherwise n_cwg per segment; plus the workgroups of a full appended region
  const int64_t new_wg_cap = ceil_div(ceil_div(capacity, a.chunk), wpw);
  if (nseg <= sgdkv::kMaxCompactSegs) {
    // the most slots and compressed-row workgroups of any call with up to new_wg_cap appended
    // workgroups per segment (appended ones count toward the rounds only while they fit in half
    // a round: past that the plan is the one without them)
    int64_t slots = 0, most = 0;
    const int64_t k_fold = std::min<int64_t>(new_wg_cap, kDecodeResident / 2 / nseg);
    for (int64_t k = 0; k <= k_fold + 1 && k <= new_wg_cap; ++k) {
      const int64_t kk = k <= k_fold ? k : new_wg_cap;
      int64_t s = 0;
      for (const int64_t n : compact_workgroups(offsets_host, nseg, a.chunk, kk)) {
        s += n + kk;
        most = std::max(most, n);
      }
      slots = std::max(slots, s);
    }
    a.n_slots = slots;
    // a segment's appended-row workgroups are numbered from n_cwg on: past its compressed-row
    // workgroups, also where whole rounds gave a segment more of them than its splits need
    a.n_cwg = (int)std::max<int64_t>(a.n_cwg, most);
  } else {
    a.n_slots = nseg * (a.n_cwg + new_wg_cap);
  }
  p.bytes = align256((size_t)a.n_slots * G * (a.D + 2) * sizeof(float));
  return SGDKV_OK;
}

}  // namespace

extern "C" {

sgdkv_status sgdkv_decode_workspace_size(const sgdkv_decode_desc* desc, const int64_t* offsets_host,
                                         size_t* bytes) {
  return sgdkv_decode_workspace_size_ex(desc, offsets_host, 0, bytes);
}

sgdkv_status sgdkv_decode_workspace_size_ex(const sgdkv_decode_desc* desc, const int64_t* offsets_host,
                                            int64_t capacity, size_t* bytes) {
  if (!bytes) return fail(SGDKV_ERR_INVALID_ARG, "NULL bytes");
  DecodePlan p;
  if (sgdkv_status st = plan_decode(desc, offsets_host, capacity, p)) return st;
  *bytes = p.bytes;
  return ok();
}

sgdkv_status sgdkv_decode_attention(const sgdkv_decode_desc* desc, const void* q, const void* k_c,
                                    const void* v_c, const int64_t* offsets, const int64_t* offsets_host,
                                    void* out, float* lse_out, void* workspace, size_t workspace_bytes,
                                    void* stream) {
  return sgdkv_decode_attention_ex(desc, q, k_c, v_c, offsets, offsets_host, nullptr, out, lse_out, workspace,
                                   workspace_bytes, stream);
}

}  // extern "C"

namespace {

// Validation and launch of one decode step, shared by the decode entry points. With
// static_scratch the split partials go to the library's static device scratch (no workspace
// argument); otherwise to the caller's workspace.
sgdkv_status decode_step(const sgdkv_decode_desc* desc, const void* q, const void* k_c, const void* v_c,
                         const int64_t* offsets, const int64_t* offsets_host, const sgdkv_decode_tail* tail,
                         void* out, float* lse_out, void* workspace, size_t workspace_bytes, bool static_scratch,
                         void* stream) {
  const sgdkv_decode_tail none{nullptr, nullptr, 0, 0};
  const sgdkv_decode_tail& t = tail ? *tail : none;
  DecodePlan p;
  if (sgdkv_status st = plan_decode(desc, offsets_host, t.capacity, p)) return st;
  sgdkv::DecodeArgs& a = p.a;
  if (t.n_new < 0 || t.n_new > t.capacity)
    return fail(SGDKV_ERR_INVALID_ARG, "n_new %lld outside [0, capacity %lld]", (long long)t.n_new,
                (long long)t.capacity);
  if (t.n_new > 0 && (!t.k_new || !t.v_new)) return fail(SGDKV_ERR_INVALID_ARG, "NULL k_new or v_new");
  if (!q || !offsets || !out) return fail(SGDKV_ERR_INVALID_ARG, "NULL q, offsets or out");
  if (a.total_rows > 0 && (!k_c || !v_c)) return fail(SGDKV_ERR_INVALID_ARG, "NULL k_c or v_c");
  const void* ptrs[] = {q, k_c, v_c, offsets, out, lse_out, t.k_new, t.v_new};
  const char* names[] = {"q", "k_c", "v_c", "offsets", "out", "lse_out", "k_new", "v_new"};
  for (int i = 0; i < 8; ++i)
    if (ptrs[i] && !aligned16(ptrs[i])) return fail(SGDKV_ERR_INVALID_ARG, "%s is not 16-byte aligned", names[i]);
  if (static_scratch) {
    if (p.bytes > sgdkv::kDecodeScratchBytes)
      return fail(SGDKV_ERR_UNSUPPORTED,
                  "this decode needs %zu bytes of split partials; the static scratch holds %zu (use "
                  "sgdkv_decode_attention_ex with a workspace)",
                  p.bytes, sgdkv::kDecodeScratchBytes);
  } else if (p.bytes > 0) {
    if (!workspace) return fail(SGDKV_ERR_WORKSPACE, "NULL workspace (%zu bytes needed)", p.bytes);
    if (reinterpret_cast<uintptr_t>(workspace) & 255u)
      return fail(SGDKV_ERR_WORKSPACE, "workspace is not 256-byte aligned");
    if (workspace_bytes < p.bytes)
      return fail(SGDKV_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", workspace_bytes, p.bytes);
  }
  if (sgdkv_status st = check_device()) return st;
  if (static_scratch) {
    hipError_t e = sgdkv::decode_scratch(&workspace);
    if (e != hipSuccess) return fail(SGDKV_ERR_HIP, "static decode scratch: %s", hipGetErrorString(e));
  }
  a.q = q;
  a.k_c = k_c;
  a.v_c = v_c;
  a.offsets = offsets;
  a.out = out;
  a.lse_out = lse_out;
  a.k_new = t.k_new;
  a.v_new = t.v_new;
  a.n_new = t.n_new;
  a.n_new_chunks = (int)ceil_div(t.n_new, a.chunk);
  a.n_new_wg = (int)ceil_div(a.n_new_chunks, sgdkv::kDecodeWaves);
  // compact decode grid: the workgroups each segment needs, from the host copy of the offsets
  const int64_t nseg = (int64_t)a.B * a.Hkv;
  a.compact = nseg <= sgdkv::kMaxCompactSegs ? 1 : 0;
  if (a.compact) {
    const std::vector<int64_t> wgs = compact_workgroups(offsets_host, nseg, a.chunk, a.n_new_wg);
    int64_t run = 0;
    a.wg_start[0] = 0;
    for (int64_t i = 0; i < nseg; ++i) {
      run += wgs[(size_t)i] + a.n_new_wg;
      a.wg_start[i + 1] = (int32_t)run;
    }
  }
  a.part = static_cast<float*>(workspace);
  a.part_ms = a.part + (size_t)a.n_slots * a.G * a.D;
  hipError_t e = hipGetLastError();
  (void)e;
  e = sgdkv::launch_decode(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(SGDKV_ERR_HIP, "decode kernels: %s", hipGetErrorString(e));
  return ok();
}

}  // namespace

extern "C" {

sgdkv_status sgdkv_decode_attention_ex(const sgdkv_decode_desc* desc, const void* q, const void* k_c,
                                       const void* v_c, const int64_t* offsets, const int64_t* offsets_host,
                                       const sgdkv_decode_tail* tail, void* out, float* lse_out, void* workspace,
                                       size_t workspace_bytes, void* stream) {
  return decode_step(desc, q, k_c, v_c, offsets, offsets_host, tail, out, lse_out, workspace, workspace_bytes,
                     false, stream);
}

sgdkv_status sgdkv_decode_attention_noalloc(const sgdkv_decode_desc* desc, const void* q, const void* k_c,
                                            const void* v_c, const int64_t* offsets, const int64_t* offsets_host,
                                            const sgdkv_decode_tail* tail, void* out, float* lse_out,
                                            void* stream) {
  return decode_step(desc, q, k_c, v_c, offsets, offsets_host, tail, out, lse_out, nullptr, 0, true, stream);
}

sgdkv_status sgdkv_append_kv(const sgdkv_decode_desc* desc, const void* k_step, const void* v_step, void* k_new,
                             void* v_new, int64_t capacity, int64_t slot, void* stream) {
  if (!desc) return fail(SGDKV_ERR_INVALID_ARG, "NULL descriptor");
  if (desc->batch < 1 || desc->num_kv_heads < 1)
    return fail(SGDKV_ERR_INVALID_ARG, "batch, num_q_heads, num_kv_heads must be >= 1");
  const int64_t nseg = (int64_t)desc->batch * desc->num_kv_heads;
  if (nseg > 65535) return fail(SGDKV_ERR_UNSUPPORTED, "batch * num_kv_heads = %lld > 65535", (long long)nseg);
  // plan with empty segments: checks the sizes and the bound of the appended region
  const std::vector<int64_t> offs((size_t)nseg + 1, 0);
  DecodePlan p;
  if (sgdkv_status st = plan_decode(desc, offs.data(), capacity, p)) return st;
  if (slot < 0 || slot >= capacity)
    return fail(SGDKV_ERR_INVALID_ARG, "slot %lld outside [0, capacity %lld)", (long long)slot, (long long)capacity);
  const void* ptrs[] = {k_step, v_step, k_new, v_new};
  const char* names[] = {"k_step", "v_step", "k_new", "v_new"};
  for (int i = 0; i < 4; ++i) {
    if (!ptrs[i]) return fail(SGDKV_ERR_INVALID_ARG, "NULL %s", names[i]);
    if (!aligned16(ptrs[i])) return fail(SGDKV_ERR_INVALID_ARG, "%s is not 16-byte aligned", names[i]);
  }
  if (sgdkv_status st = check_device()) return st;
  hipError_t e = hipGetLastError();
  (void)e;
  e = sgdkv::launch_append(p.a, k_step, v_step, k_new, v_new, slot, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(SGDKV_ERR_HIP, "append kernel: %s", hipGetErrorString(e));
  return ok();
}

}  // extern "C"
