// Host-side parts of the ABI: error state, token budget, the offline SLC
// policy (Eq. 5), the admission rule of Algorithm 1 / Eq. 6, and the
// kernel-class profiler.  Built with -ffp-contract=off so that the double
// arithmetic of the policy and the plan rounds after every operation.
#include <cmath>
#include <mutex>
#include <vector>

#include "common.h"

namespace spider {

static thread_local std::string g_error;

void set_error(const char* fmt, ...) {
  char buf[1024];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_error = buf;
}

void clear_error() { g_error.clear(); }

// ----------------------------------------------------------------- profiler
namespace {
struct ProfRecord {
  int cls;
  hipEvent_t start, stop;
};
struct Profiler {
  bool enabled = false;
  uint32_t mask = 0xFFFFFFFFu;
  std::vector<ProfRecord> records;
  std::vector<hipEvent_t> pool;
  int64_t launches[KC_COUNT] = {};
  double total_ms[KC_COUNT] = {};
  std::vector<int> open;  // index into records of the currently open scope per class
};
Profiler g_prof;
std::mutex g_prof_mu;

hipEvent_t take_event() {
  if (!g_prof.pool.empty()) {
    hipEvent_t e = g_prof.pool.back();
    g_prof.pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void drain_records() {
  for (auto& r : g_prof.records) {
    if (r.start && r.stop && hipEventSynchronize(r.stop) == hipSuccess) {
      float ms = 0.f;
      if (hipEventElapsedTime(&ms, r.start, r.stop) == hipSuccess) {
        g_prof.launches[r.cls] += 1;
        g_prof.total_ms[r.cls] += ms;
      }
    }
    if (r.start) g_prof.pool.push_back(r.start);
    if (r.stop) g_prof.pool.push_back(r.stop);
  }
  g_prof.records.clear();
}

const char* kClassNames[KC_COUNT] = {
    "score_prep", "anchor_topk", "kmeans",   "anchor_maxsim", "score_final",
    "select",     "assemble",    "embed",    "rmsnorm",       "gemm_qkv",
    "qkv_finalize", "attention", "gemm_o",   "gemm_gateup",   "gemm_down",
    "residual_add", "lens_prep", "gemm_lens", "lens_admit", "anchor_colmean", "cls_attention", "projector", "lm_head"};
}  // namespace

void prof_begin(int cls, hipStream_t s) {
  if (!g_prof.enabled || !((g_prof.mask >> cls) & 1u)) return;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  ProfRecord r{cls, take_event(), nullptr};
  if (r.start) hipEventRecord(r.start, s);
  g_prof.records.push_back(r);
  if ((int)g_prof.open.size() < KC_COUNT) g_prof.open.assign(KC_COUNT, -1);
  g_prof.open[cls] = (int)g_prof.records.size() - 1;
  if (g_prof.records.size() > 4096) {
    // keep memory bounded: fold finished records into the totals
    std::vector<ProfRecord> keep;
    for (size_t i = 0; i + 1 < g_prof.records.size(); ++i) {
      auto& q = g_prof.records[i];
      if (q.stop) {
        if (hipEventSynchronize(q.stop) == hipSuccess) {
          float ms = 0.f;
          if (hipEventElapsedTime(&ms, q.start, q.stop) == hipSuccess) {
            g_prof.launches[q.cls] += 1;
            g_prof.total_ms[q.cls] += ms;
          }
        }
        g_prof.pool.push_back(q.start);
        g_prof.pool.push_back(q.stop);
      } else {
        keep.push_back(q);
      }
    }
    keep.push_back(g_prof.records.back());
    g_prof.records.swap(keep);
    g_prof.open.assign(KC_COUNT, -1);
    g_prof.open[cls] = (int)g_prof.records.size() - 1;
  }
}

void prof_end(int cls, hipStream_t s) {
  if (!g_prof.enabled || !((g_prof.mask >> cls) & 1u)) return;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if ((int)g_prof.open.size() < KC_COUNT) return;
  int i = g_prof.open[cls];
  if (i < 0 || i >= (int)g_prof.records.size()) return;
  hipEvent_t e = take_event();
  if (e) hipEventRecord(e, s);
  g_prof.records[i].stop = e;
  g_prof.open[cls] = -1;
}

}  // namespace spider

using namespace spider;

extern "C" {

const char* spider_last_error(void) { return g_error.c_str(); }

int spider_version(void) { return 101; }

spider_status spider_budget(int keep, int r_num, int r_den, int* n_anchor, int* n_cmp) {
  clear_error();
  SPIDER_REQUIRE(n_anchor && n_cmp, SPIDER_ERR_INVALID_ARG, "spider_budget: null output");
  SPIDER_REQUIRE(keep >= 0 && r_den > 0 && r_num >= 0 && r_num <= r_den, SPIDER_ERR_INVALID_ARG,
                 "spider_budget: need keep >= 0, r_den > 0, 0 <= r_num <= r_den");
  long long k = (long long)keep * r_num / r_den;
  *n_anchor = (int)k;
  *n_cmp = keep - (int)k;
  return SPIDER_OK;
}

spider_status spider_budget_ratio(int n, int rv_num, int rv_den, int r_num, int r_den, int* keep,
                                  int* n_anchor, int* n_cmp) {
  clear_error();
  SPIDER_REQUIRE(keep && n_anchor && n_cmp, SPIDER_ERR_INVALID_ARG, "spider_budget_ratio: null output");
  SPIDER_REQUIRE(n >= 0 && rv_den > 0 && rv_num >= 0 && rv_num <= rv_den, SPIDER_ERR_INVALID_ARG,
                 "spider_budget_ratio: need n >= 0, rv_den > 0, 0 <= rv_num <= rv_den");
  const int kp = (int)((long long)n * rv_num / rv_den);
  int a = 0, c = 0;
  const spider_status s = spider_budget(kp, r_num, r_den, &a, &c);
  if (s != SPIDER_OK) return s;
  *keep = kp;
  *n_anchor = a;
  *n_cmp = c;
  return SPIDER_OK;
}

spider_status spider_slc_policy(int L, const float* slc_attn, const float* slc_ffn, double eps,
                                double* slc_sel_out, uint8_t* target_out) {
  clear_error();
  SPIDER_REQUIRE(L >= 1, SPIDER_ERR_INVALID_ARG, "spider_slc_policy: L must be >= 1");
  SPIDER_REQUIRE(slc_attn && slc_ffn && slc_sel_out && target_out, SPIDER_ERR_INVALID_ARG,
                 "spider_slc_policy: null pointer");
  SPIDER_REQUIRE(eps >= 0.0, SPIDER_ERR_INVALID_ARG, "spider_slc_policy: eps must be >= 0");
  const float* fam[2] = {slc_attn, slc_ffn};
  std::vector<double> norm[2];
  for (int f = 0; f < 2; ++f) {
    double lo = (double)fam[f][0], hi = (double)fam[f][0];
    for (int l = 1; l < L; ++l) {
      double v = (double)fam[f][l];
      if (v < lo) lo = v;
      if (v > hi) hi = v;
    }
    for (int l = 0; l < L; ++l) {
      SPIDER_REQUIRE(std::isfinite(fam[f][l]), SPIDER_ERR_INVALID_ARG,
                     "spider_slc_policy: non-finite score at layer %d", l);
    }
    double den = (hi - lo) + eps;
    norm[f].resize(L);
    for (int l = 0; l < L; ++l) {
      double num = (double)fam[f][l] - lo;
      norm[f][l] = (den > 0.0) ? 1.0 - num / den : 1.0;
    }
  }
  for (int l = 0; l < L; ++l) {
    bool ffn = norm[1][l] > norm[0][l];
    target_out[l] = ffn ? 1 : 0;
    slc_sel_out[l] = ffn ? norm[1][l] : norm[0][l];
  }
  return SPIDER_OK;
}

spider_status spider_plan_skips(int L, int n_vis, const float* s_sa, int s_sa_stride,
                                const double* slc_sel, const uint8_t* target, double w1, double w2,
                                double T_skip, uint8_t* codes_out, int codes_stride,
                                int32_t* admit_out) {
  clear_error();
  SPIDER_REQUIRE(L >= 1 && n_vis >= 0, SPIDER_ERR_INVALID_ARG,
                 "spider_plan_skips: need L >= 1 and n_vis >= 0");
  SPIDER_REQUIRE(slc_sel && target && codes_out, SPIDER_ERR_INVALID_ARG,
                 "spider_plan_skips: null pointer");
  const int W = L / 2;
  SPIDER_REQUIRE(W == 0 || n_vis == 0 || s_sa, SPIDER_ERR_INVALID_ARG,
                 "spider_plan_skips: s_sa is null");
  SPIDER_REQUIRE(s_sa_stride >= n_vis && codes_stride >= n_vis, SPIDER_ERR_SHAPE,
                 "spider_plan_skips: strides must be >= n_vis");
  for (int l = 0; l < L; ++l)
    SPIDER_REQUIRE(target[l] <= 1, SPIDER_ERR_INVALID_ARG,
                   "spider_plan_skips: target[%d] must be 0 or 1", l);
  std::vector<double> acc(n_vis, 0.0);
  std::vector<int> admit(n_vis, -1);
  for (int l = 0; l < W; ++l) {
    const double sel = slc_sel[l];
    for (int i = 0; i < n_vis; ++i) {
      if (admit[i] >= 0) continue;
      const double fuse = w1 * (double)s_sa[(size_t)l * s_sa_stride + i] + w2 * sel;
      acc[i] = acc[i] + fuse;
      if (acc[i] >= T_skip) admit[i] = l;
    }
  }
  for (int l = 0; l < L; ++l)
    for (int i = 0; i < n_vis; ++i) {
      uint8_t c = 0;
      if (admit[i] >= 0 && l >= admit[i]) c = target[admit[i]] ? 2 : 1;
      codes_out[(size_t)l * codes_stride + i] = c;
    }
  if (admit_out)
    for (int i = 0; i < n_vis; ++i) admit_out[i] = admit[i];
  return SPIDER_OK;
}

spider_status spider_profile_enable(int enable) {
  clear_error();
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (enable) {
    drain_records();
    for (int i = 0; i < KC_COUNT; ++i) {
      g_prof.launches[i] = 0;
      g_prof.total_ms[i] = 0.0;
    }
    g_prof.open.assign(KC_COUNT, -1);
    g_prof.enabled = true;
  } else {
    g_prof.enabled = false;
  }
  return SPIDER_OK;
}

spider_status spider_profile_mask(uint32_t mask) {
  clear_error();
  std::lock_guard<std::mutex> lk(g_prof_mu);
  drain_records();
  g_prof.mask = mask;
  return SPIDER_OK;
}

int spider_profile_classes(void) { return KC_COUNT; }

const char* spider_profile_class_name(int cls) {
  if (cls < 0 || cls >= KC_COUNT) return "";
  return kClassNames[cls];
}

spider_status spider_profile_read(int cls, int64_t* launches, double* total_ms) {
  clear_error();
  SPIDER_REQUIRE(cls >= 0 && cls < KC_COUNT, SPIDER_ERR_INVALID_ARG,
                 "spider_profile_read: class out of range");
  SPIDER_REQUIRE(launches && total_ms, SPIDER_ERR_INVALID_ARG, "spider_profile_read: null output");
  std::lock_guard<std::mutex> lk(g_prof_mu);
  drain_records();
  *launches = g_prof.launches[cls];
  *total_ms = g_prof.total_ms[cls];
  return SPIDER_OK;
}

}  // extern "C"
