// Host-side sanitizer run: the C-ABI host layer (budget allocation, offsets,
// argument validation of the device entry points) and the CPU oracle, built
// together with AddressSanitizer and UndefinedBehaviorSanitizer, exercised on
// seeded random problems. Allocation results of the two are compared; the
// device entry points are driven through their validation paths only (with no
// usable device they stop with SGDKV_ERR_HIP after validation).
//
// Test infrastructure: built and run by tests/test_sanitize_host.py.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "sgdkv.h"

extern "C" {
int orc_reduce_group_max(const double* per_q, int L, int Hq, int Hkv, double* out);
int orc_total_from_ratio(double R, int L, int H, int64_t C, int64_t s, int64_t W, int of_middle, int64_t* out);
int orc_allocate_budgets(const double* sigma, int L, int H, int64_t C, int64_t s, int64_t W, int64_t total, int mode,
                         int64_t* out);
int orc_allocate_variant(const double* sigma, const double* sigma2, int L, int H, int64_t C, int64_t s, int64_t W,
                         int64_t total, int mode, int variant, double full_fraction, int64_t* out);
int orc_window_lse(const double* q_win, const double* k, int B, int Hq, int Hkv, int d, int64_t C, int w,
                   int64_t win0, double scale, double* lse);
int orc_window_colsum(const double* q_win, const double* k, const double* lse, int B, int Hq, int Hkv, int d,
                      int64_t C, int w, int64_t win0, double scale, double* colsum);
int orc_window_colsum_ipt(const double* q_win, const double* k, const double* lse, int B, int Hq, int Hkv, int d,
                          int64_t C, int w, int64_t win0, double scale, const double* qscores, int agg,
                          double* colsum);
int orc_pool(const double* a, int64_t rows, int64_t n, int kp, double* pooled);
int orc_select(const double* pooled, int64_t C, int64_t n_scored, int64_t s, int64_t W, int64_t m, int32_t* kept);
int orc_decode(const double* q, const double* kc, const double* vc, const int64_t* offsets, int B, int Hq, int Hkv,
               int d, double scale, double* out, double* lse);
int orc_decode_append(const double* q, const double* kc, const double* vc, const int64_t* offsets,
                      const double* k_new, const double* v_new, int64_t cap, int64_t n_new, int B, int Hq, int Hkv,
                      int d, double scale, double* out, double* lse);
}

namespace {

uint64_t g_state = 0x9E3779B97F4A7C15ull;
uint64_t next_u64() {  // xorshift64*
  g_state ^= g_state >> 12;
  g_state ^= g_state << 25;
  g_state ^= g_state >> 27;
  return g_state * 0x2545F4914F6CDD1Dull;
}
double uniform() { return (double)(next_u64() >> 11) * (1.0 / 9007199254740992.0); }
int64_t randint(int64_t lo, int64_t hi) { return lo + (int64_t)(next_u64() % (uint64_t)(hi - lo + 1)); }
double normal() {
  const double u = uniform() + 1e-300, v = uniform();
  return std::sqrt(-2.0 * std::log(u)) * std::cos(6.283185307179586 * v);
}

int g_failures = 0;
void expect(bool ok, const char* what, long long a = 0, long long b = 0) {
  if (!ok) {
    ++g_failures;
    std::fprintf(stderr, "FAIL: %s (%lld, %lld): %s\n", what, a, b, sgdkv_last_error());
  }
}

void allocation_against_oracle(int rounds) {
  for (int r = 0; r < rounds; ++r) {
    const int L = (int)randint(1, 4), H = (int)randint(1, 8), n = L * H;
    const int64_t C = randint(1, 5000), s = randint(0, 64), W = randint(0, 64);
    std::vector<double> sc(n), sc2(n);
    const int kind = (int)randint(0, 3);
    for (int h = 0; h < n; ++h) {
      sc[h] = kind == 0 ? uniform() : kind == 1 ? uniform() * 1e6 : kind == 2 ? (double)randint(0, 2) * 0.5 : 0.0;
      sc2[h] = uniform();
    }
    if (s + W > C) {
      std::vector<int64_t> out(n, -7);
      expect(sgdkv_allocate_budgets(sc.data(), L, H, C, s, W, n * C, 0, out.data()) == SGDKV_ERR_INVALID_ARG,
             "s + W > C rejected");
      expect(out[0] == -7, "nothing written on error");
      continue;
    }
    const int64_t total = n * (s + W) + (int64_t)std::floor(uniform() * (double)(n * (C - s - W)));
    for (int mode = 0; mode < 2; ++mode) {
      std::vector<int64_t> got(n), ref(n);
      expect(sgdkv_allocate_budgets(sc.data(), L, H, C, s, W, total, mode, got.data()) == SGDKV_OK, "allocate");
      expect(orc_allocate_budgets(sc.data(), L, H, C, s, W, total, mode, ref.data()) == 0, "oracle allocate");
      int64_t sum = 0;
      for (int h = 0; h < n; ++h) {
        expect(got[h] == ref[h], "budget equals the oracle's", got[h], ref[h]);
        expect(got[h] >= s + W && got[h] <= C, "budget in range", got[h], C);
        sum += got[h];
      }
      expect(sum == total, "budgets sum to the total", sum, total);
      for (int variant = 0; variant <= 5; ++variant) {
        const double f = uniform();
        std::vector<int64_t> gv(n), rv(n);
        const int st = sgdkv_allocate_budgets_variant(sc.data(), sc2.data(), L, H, C, s, W, total, mode, variant, f,
                                                      gv.data());
        const int so = orc_allocate_variant(sc.data(), sc2.data(), L, H, C, s, W, total, mode, variant, f, rv.data());
        expect(st == SGDKV_OK && so == 0, "variant status", st, so);
        for (int h = 0; h < n; ++h) expect(gv[h] == rv[h], "variant budget equals the oracle's", gv[h], rv[h]);
      }
    }
    int64_t t_lib = 0, t_orc = 0;
    const double R = uniform();
    const int st = sgdkv_total_from_ratio(R, L, H, C, s, W, 1, &t_lib);
    const int so = orc_total_from_ratio(R, L, H, C, s, W, 1, &t_orc);
    expect(st == SGDKV_OK && so == 0 && t_lib == t_orc, "total_from_ratio", t_lib, t_orc);
    // GQA reduction
    const int G = (int)randint(1, 4);
    std::vector<double> pq((size_t)L * H * G), red(n), ored(n);
    for (double& x : pq) x = uniform();
    expect(sgdkv_reduce_query_head_scores(pq.data(), L, H * G, H, red.data()) == SGDKV_OK, "reduce");
    expect(orc_reduce_group_max(pq.data(), L, H * G, H, ored.data()) == 0, "oracle reduce");
    for (int h = 0; h < n; ++h) expect(red[h] == ored[h], "reduced score equals the oracle's");
  }
}

void offsets_cases(int rounds) {
  for (int r = 0; r < rounds; ++r) {
    const int B = (int)randint(1, 40), H = (int)randint(1, 64);
    std::vector<int64_t> bud(H), off((size_t)B * H + 1, -1);
    for (int64_t& x : bud) x = randint(0, 1 << 20);
    expect(sgdkv_segment_offsets(bud.data(), B, H, off.data()) == SGDKV_OK, "segment offsets");
    int64_t row = 0;
    for (int b = 0; b < B; ++b)
      for (int h = 0; h < H; ++h) {
        expect(off[(size_t)b * H + h] == row, "segment start", off[(size_t)b * H + h], row);
        row += bud[h];
      }
    expect(off[(size_t)B * H] == row, "total rows");
  }
  int64_t bad[2] = {1, -1}, out[5] = {-7, -7, -7, -7, -7};
  expect(sgdkv_segment_offsets(bad, 2, 2, out) == SGDKV_ERR_INVALID_ARG && out[0] == -7, "negative budget");
  expect(sgdkv_segment_offsets(nullptr, 2, 2, out) == SGDKV_ERR_INVALID_ARG, "NULL budgets");
}

void device_validation() {
  // fake, aligned device addresses: validation rejects or the (absent) device does
  void* F = reinterpret_cast<void*>(uintptr_t(1) << 40);
  char* Fc = static_cast<char*>(F);
  sgdkv_compress_desc d{2, 4, 2, 64, 32, 7, 2048, 4, 32, SGDKV_DTYPE_F32, 0.f};
  size_t ws = 0;
  expect(sgdkv_compress_workspace_size(&d, &ws) == SGDKV_OK && ws > 0, "compress workspace size");
  const int64_t bud[2] = {512, 512};
  auto compress = [&](const sgdkv_compress_desc& dd, const int64_t* b, size_t wsb, void* kout) {
    return sgdkv_compress_layer(&dd, b, F, F, F, nullptr, kout, F, static_cast<int32_t*>(F),
                                static_cast<int64_t*>(F), static_cast<float*>(F), F, wsb, nullptr);
  };
  const int none = compress(d, bud, ws, F);
  expect(none == SGDKV_ERR_HIP || none == SGDKV_OK, "well-formed compress reaches the device check", none);
  sgdkv_compress_desc e = d;
  e.pool_kernel = 4;
  expect(compress(e, bud, ws, F) == SGDKV_ERR_INVALID_ARG, "even pool kernel");
  e = d;
  e.head_dim = 80;
  expect(compress(e, bud, ws, F) == SGDKV_ERR_UNSUPPORTED, "head_dim 80");
  e = d;
  e.b_window = 8;
  expect(compress(e, bud, ws, F) == SGDKV_ERR_INVALID_ARG, "b_window < obs_window");
  const int64_t badbud[2] = {10, 512};
  expect(compress(d, badbud, ws, F) == SGDKV_ERR_INVALID_ARG, "budget below s + W");
  expect(compress(d, bud, ws - 1, F) == SGDKV_ERR_WORKSPACE, "small workspace");
  expect(compress(d, bud, ws, Fc + 8) == SGDKV_ERR_INVALID_ARG, "misaligned output");
  sgdkv_compress_opts o{SGDKV_GROUP_IPT_MAX, 0, nullptr, -1, nullptr};
  expect(sgdkv_compress_layer_ex(&d, &o, bud, F, F, F, nullptr, F, F, static_cast<int32_t*>(F),
                                 static_cast<int64_t*>(F), nullptr, F, ws, nullptr) == SGDKV_ERR_INVALID_ARG,
         "Ipt. without scores");

  sgdkv_decode_desc dd{2, 4, 2, 64, 1, 0, 0.f};
  const int64_t oh[5] = {0, 10, 10, 30, 31};
  size_t dws = 0;
  expect(sgdkv_decode_workspace_size(&dd, oh, &dws) == SGDKV_OK, "decode workspace size");
  auto decode = [&](const sgdkv_decode_desc& x, const int64_t* offs, size_t wsb) {
    return sgdkv_decode_attention(&x, F, F, F, static_cast<int64_t*>(F), offs, F, nullptr, F, wsb, nullptr);
  };
  const int dn = decode(dd, oh, dws);
  expect(dn == SGDKV_ERR_HIP || dn == SGDKV_OK, "well-formed decode reaches the device check", dn);
  const int64_t dec[5] = {0, 10, 9, 30, 31};
  expect(decode(dd, dec, dws) == SGDKV_ERR_INVALID_ARG, "decreasing offsets");
  sgdkv_decode_desc big = dd;
  big.num_q_heads = 34;
  expect(decode(big, oh, dws) == SGDKV_ERR_UNSUPPORTED, "group of 17");
  expect(decode(dd, oh, 8) == SGDKV_ERR_WORKSPACE, "small decode workspace");
  sgdkv_decode_tail t{F, F, 100, 101};
  expect(sgdkv_decode_attention_ex(&dd, F, F, F, static_cast<int64_t*>(F), oh, &t, F, nullptr, F, dws, nullptr) ==
             SGDKV_ERR_INVALID_ARG,
         "n_new > capacity");
  expect(sgdkv_append_kv(&dd, F, F, F, F, 10, 10, nullptr) == SGDKV_ERR_INVALID_ARG, "slot == capacity");
}

// Decode planning over ragged segment sets: empty, one-row and long segments, past one round of
// decode workgroups (their share-out over the segments) and within it, with appended regions.
void decode_plans(int rounds) {
  for (int r = 0; r < rounds; ++r) {
    const int Hkv = (int)randint(1, 8), B = (int)randint(1, 512 / Hkv), G = (int)randint(1, 16);
    const int64_t nseg = (int64_t)B * Hkv;
    std::vector<int64_t> oh((size_t)nseg + 1, 0);
    const int64_t top = randint(0, 3) == 0 ? 3000 : (int64_t)1 << randint(10, 20);
    for (int64_t i = 0; i < nseg; ++i) {
      const int kind = (int)randint(0, 9);
      const int64_t len = kind == 0 ? 0 : kind == 1 ? 1 : kind == 2 ? randint(2, 40) : randint(0, top);
      oh[(size_t)i + 1] = oh[(size_t)i] + len;
    }
    sgdkv_decode_desc dd{B, Hkv * G, Hkv, randint(0, 1) ? 128 : 64, (int)randint(0, 1), 0, 0.f};
    size_t bytes = 0;
    const int64_t cap = randint(0, 2) == 0 ? randint(1, 300) : 0;
    expect(sgdkv_decode_workspace_size_ex(&dd, oh.data(), cap, &bytes) == SGDKV_OK, "decode plan", r);
    int64_t nonempty = 0;
    for (int64_t i = 0; i < nseg; ++i) nonempty += oh[(size_t)i + 1] > oh[(size_t)i];
    const size_t per_wg = (size_t)G * (dd.head_dim + 2) * sizeof(float);
    expect(bytes >= (size_t)nonempty * per_wg, "a workgroup slot per non-empty segment", r);
  }
}

void oracle_compress_decode(int rounds) {
  for (int r = 0; r < rounds; ++r) {
    const int B = (int)randint(1, 2), Hkv = (int)randint(1, 3), G = (int)randint(1, 3), Hq = Hkv * G;
    const int d = 8 * (int)randint(1, 4);
    const int64_t C = randint(40, 300);
    const int w = (int)randint(1, 16);
    const int64_t s = randint(0, 5), W = randint(w, 24);
    const int64_t win0 = C - w;
    const int kp = 2 * (int)randint(0, 3) + 1;
    std::vector<double> q((size_t)B * Hq * w * d), k((size_t)B * Hkv * C * d), lse((size_t)B * Hq * w);
    std::vector<double> col((size_t)B * Hkv * win0), pooled((size_t)B * Hkv * win0), qs(Hq);
    for (double& x : q) x = normal();
    for (double& x : k) x = normal();
    for (double& x : qs) x = uniform();
    expect(orc_window_lse(q.data(), k.data(), B, Hq, Hkv, d, C, w, win0, 1.0 / std::sqrt((double)d), lse.data()) == 0, "oracle lse");
    expect(orc_window_colsum(q.data(), k.data(), lse.data(), B, Hq, Hkv, d, C, w, win0, 1.0 / std::sqrt((double)d), col.data()) == 0,
           "oracle colsum");
    for (int agg = 1; agg <= 3; ++agg)
      expect(orc_window_colsum_ipt(q.data(), k.data(), lse.data(), B, Hq, Hkv, d, C, w, win0, 1.0 / std::sqrt((double)d), qs.data(), agg,
                                   col.data()) == 0,
             "oracle Ipt. colsum");
    expect(orc_window_colsum(q.data(), k.data(), lse.data(), B, Hq, Hkv, d, C, w, win0, 1.0 / std::sqrt((double)d), col.data()) == 0,
           "oracle colsum");
    expect(orc_pool(col.data(), (int64_t)B * Hkv, win0, kp, pooled.data()) == 0, "oracle pool");
    std::vector<int64_t> offs((size_t)B * Hkv + 1, 0);
    std::vector<int32_t> kept;
    int64_t row = 0;
    for (int b = 0; b < B; ++b)
      for (int h = 0; h < Hkv; ++h) {
        const int64_t m = randint(0, C - s - W);
        std::vector<int32_t> seg((size_t)(s + W + m));
        expect(orc_select(&pooled[((size_t)b * Hkv + h) * win0], C, win0, s, W, m, seg.data()) == 0, "select");
        for (size_t i = 1; i < seg.size(); ++i) expect(seg[i - 1] < seg[i], "kept rows ascending");
        offs[(size_t)b * Hkv + h] = row;
        row += (int64_t)seg.size();
        kept.insert(kept.end(), seg.begin(), seg.end());
      }
    offs[(size_t)B * Hkv] = row;
    std::vector<double> kc((size_t)row * d), vc((size_t)row * d), qd((size_t)B * Hq * d), out((size_t)B * Hq * d),
        dl((size_t)B * Hq);
    for (double& x : kc) x = normal();
    for (double& x : vc) x = normal();
    for (double& x : qd) x = normal();
    expect(orc_decode(qd.data(), kc.data(), vc.data(), offs.data(), B, Hq, Hkv, d, 0.0, out.data(), dl.data()) == 0,
           "oracle decode");
    const int64_t cap = randint(0, 5), n_new = randint(0, cap);
    std::vector<double> kn((size_t)B * Hkv * cap * d + 1), vn((size_t)B * Hkv * cap * d + 1);
    for (double& x : kn) x = normal();
    for (double& x : vn) x = normal();
    expect(orc_decode_append(qd.data(), kc.data(), vc.data(), offs.data(), kn.data(), vn.data(), cap, n_new, B, Hq,
                             Hkv, d, 0.0, out.data(), dl.data()) == 0,
           "oracle decode with appended rows");
  }
}

}  // namespace

int main() {
  allocation_against_oracle(400);
  offsets_cases(100);
  device_validation();
  decode_plans(300);
  oracle_compress_decode(40);
  if (g_failures) {
    std::fprintf(stderr, "%d failures\n", g_failures);
    return 1;
  }
  std::printf("SANITIZE PASS\n");
  return 0;
}
