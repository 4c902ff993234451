// Error state, profiler and small host helpers of libkronq.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <string>
#include <utility>
#include <vector>

#include "kq_common.hpp"

namespace kq {

namespace {
thread_local char g_err[512] = "";

struct ProfEntry {
  std::vector<std::pair<hipEvent_t, hipEvent_t>> pending;
  double ms = 0.0;
  int64_t launches = 0;
};
bool g_prof = false;
std::string g_prof_only;  // empty: every kernel; else only kernels with exactly this name
std::map<std::string, ProfEntry> g_prof_tab;
std::vector<hipEvent_t> g_event_pool;
hipEvent_t g_open = nullptr;

hipEvent_t take_event() {
  if (!g_event_pool.empty()) {
    hipEvent_t e = g_event_pool.back();
    g_event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void drain(ProfEntry& p) {
  for (auto& ev : p.pending) {
    float ms = 0.f;
    if (ev.first && ev.second && hipEventSynchronize(ev.second) == hipSuccess &&
        hipEventElapsedTime(&ms, ev.first, ev.second) == hipSuccess) {
      p.ms += ms;
      p.launches += 1;
    }
    if (ev.first) g_event_pool.push_back(ev.first);
    if (ev.second) g_event_pool.push_back(ev.second);
  }
  p.pending.clear();
}
}  // namespace

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
}

void clear_error() { g_err[0] = '\0'; }

bool prof_on() { return g_prof; }

// g_prof_only: empty (every kernel), or kernel names separated by commas
bool prof_wants(const char* name) {
  if (g_prof_only.empty()) return true;
  const std::string n(name);
  size_t b = 0;
  while (b <= g_prof_only.size()) {
    size_t e = g_prof_only.find(',', b);
    if (e == std::string::npos) e = g_prof_only.size();
    if (g_prof_only.compare(b, e - b, n) == 0 && e - b == n.size()) return true;
    b = e + 1;
  }
  return false;
}

void prof_begin(const char* name, hipStream_t s) {
  (void)name;
  g_open = take_event();
  if (g_open) (void)hipEventRecord(g_open, s);
}

void prof_end(const char* name, hipStream_t s) {
  hipEvent_t stop = take_event();
  if (stop) (void)hipEventRecord(stop, s);
  g_prof_tab[name].pending.emplace_back(g_open, stop);
  g_open = nullptr;
}

RotDim rot_dim(int64_t d) {
  RotDim r;
  auto pow2 = [](int64_t x) { return x > 0 && (x & (x - 1)) == 0; };
  if (d >= 2 && pow2(d)) {
    r.ok = true;
    r.m = d;
  } else if (d % 28 == 0 && pow2(d / 28) && d / 28 <= 16384) {
    r.ok = true;
    r.has28 = true;
    r.m = d / 28;
  }
  return r;
}

}  // namespace kq

extern "C" {

const char* kronq_last_error(void) { return kq::g_err; }

int kronq_version(void) { return 100; }

int kronq_profile_enable(int on) {
  kq::g_prof = on != 0;
  return KRONQ_OK;
}

int kronq_profile_only(const char* kernel) {
  kq::g_prof_only = kernel ? kernel : "";
  return KRONQ_OK;
}

void kronq_profile_reset(void) {
  for (auto& kv : kq::g_prof_tab) {
    kq::drain(kv.second);
  }
  kq::g_prof_tab.clear();
}

int kronq_profile_read(const char* kernel, double* total_ms, int64_t* launches) {
  KQ_REQUIRE(kernel && total_ms && launches, KRONQ_ERR_INVALID_ARG, "null argument");
  auto it = kq::g_prof_tab.find(kernel);
  if (it == kq::g_prof_tab.end()) {
    *total_ms = 0.0;
    *launches = 0;
    return KRONQ_OK;
  }
  kq::drain(it->second);
  *total_ms = it->second.ms;
  *launches = it->second.launches;
  return KRONQ_OK;
}

int64_t kronq_profile_names(char* buf, size_t cap) {
  std::string all;
  for (const auto& kv : kq::g_prof_tab) {
    if (!all.empty()) all += ',';
    all += kv.first;
  }
  if (buf && cap > 0) {
    const size_t n = all.size() < cap - 1 ? all.size() : cap - 1;
    std::memcpy(buf, all.data(), n);
    buf[n] = '\0';
  }
  return static_cast<int64_t>(all.size());
}

int kronq_allocate_bits(const double* scores, const int64_t* weights, int n_layers,
                        const int* choices, int n_choices, double avg_bits, int* bits_out,
                        double* objective_out) {
  KQ_REQUIRE(scores && weights && choices && bits_out, KRONQ_ERR_INVALID_ARG, "null argument");
  KQ_REQUIRE(n_layers >= 1 && n_layers <= 12 && n_choices >= 1 && n_choices <= 8,
             KRONQ_ERR_INVALID_ARG, "n_layers must be in [1,12] and n_choices in [1,8]");
  int ch[8];
  for (int i = 0; i < n_choices; ++i) {
    KQ_REQUIRE(choices[i] >= 1 && choices[i] <= 16, KRONQ_ERR_INVALID_ARG, "bad bit choice");
    ch[i] = choices[i];
  }
  for (int i = 1; i < n_choices; ++i)  // insertion sort: lexicographic order of sorted choices
    for (int j = i; j > 0 && ch[j - 1] > ch[j]; --j) std::swap(ch[j - 1], ch[j]);
  int64_t wsum = 0;
  for (int l = 0; l < n_layers; ++l) {
    KQ_REQUIRE(weights[l] >= 0, KRONQ_ERR_INVALID_ARG, "negative weight");
    wsum += weights[l];
  }
  const double budget = avg_bits * static_cast<double>(wsum);
  int idx[12] = {0};
  int best[12];
  double best_val = 0.0;
  bool found = false;
  while (true) {
    int64_t used = 0;
    for (int l = 0; l < n_layers; ++l) used += weights[l] * ch[idx[l]];
    if (static_cast<double>(used) <= budget) {
      double val = 0.0;
      for (int l = 0; l < n_layers; ++l) {
        const double q = static_cast<double>((1LL << ch[idx[l]]) - 1);
        val += scores[l] / (q * q);
      }
      if (!found || val < best_val) {
        found = true;
        best_val = val;
        for (int l = 0; l < n_layers; ++l) best[l] = ch[idx[l]];
      }
    }
    int l = n_layers - 1;  // next vector in lexicographic order (last position fastest)
    while (l >= 0 && idx[l] == n_choices - 1) {
      idx[l] = 0;
      --l;
    }
    if (l < 0) break;
    ++idx[l];
  }
  KQ_REQUIRE(found, KRONQ_ERR_SHAPE, "no assignment meets the bit budget");
  for (int l = 0; l < n_layers; ++l) bits_out[l] = best[l];
  if (objective_out) *objective_out = best_val;
  return KRONQ_OK;
}

}  // extern "C"
