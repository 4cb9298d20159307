// Per-kernel HIP-event timing (see prof.h). Events are recycled through a
// pool; querying synchronises on the recorded events only.
#include "prof.h"

#include <string.h>

#include <mutex>
#include <string>
#include <vector>

#include "rnnt_pruned.h"

namespace {

struct Rec {
  std::string name;
  hipEvent_t a, b;
  bool closed;
};

std::mutex g_mu;
bool g_on = false;
std::vector<Rec> g_recs;
std::vector<hipEvent_t> g_pool;
std::vector<std::string> g_sel;  // names to record; empty: all

bool selected(const char* name) {
  if (g_sel.empty()) return true;
  for (auto& s : g_sel)
    if (s == name) return true;
  return false;
}

hipEvent_t get_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

}  // namespace

void prof_begin(hipStream_t s, const char* name) {
  if (!g_on) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!selected(name)) return;
  hipEvent_t a = get_event(), b = get_event();
  if (!a || !b) return;
  hipEventRecord(a, s);
  g_recs.push_back(Rec{name, a, b, false});
}

void prof_end(hipStream_t s, const char* name) {
  if (!g_on) return;
  std::lock_guard<std::mutex> lk(g_mu);
  for (auto it = g_recs.rbegin(); it != g_recs.rend(); ++it) {
    if (!it->closed && it->name == name) {
      hipEventRecord(it->b, s);
      it->closed = true;
      return;
    }
  }
}

extern "C" {

int rnnt_profile_enable(int on) {
  std::lock_guard<std::mutex> lk(g_mu);
  g_on = on != 0;
  return RNNT_OK;
}

int rnnt_profile_select(const char* names) {
  std::lock_guard<std::mutex> lk(g_mu);
  g_sel.clear();
  if (!names) return RNNT_OK;
  std::string cur;
  for (const char* c = names;; ++c) {
    if (*c == ',' || *c == 0) {
      if (!cur.empty()) g_sel.push_back(cur);
      cur.clear();
      if (*c == 0) break;
    } else {
      cur += *c;
    }
  }
  return RNNT_OK;
}

int rnnt_profile_reset(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  for (auto& r : g_recs) {
    hipEventSynchronize(r.b);
    g_pool.push_back(r.a);
    g_pool.push_back(r.b);
  }
  g_recs.clear();
  return RNNT_OK;
}

int rnnt_profile_query(const char* name, int32_t* launches, double* total_ms) {
  if (!name || !launches || !total_ms) return RNNT_EINVAL;
  std::lock_guard<std::mutex> lk(g_mu);
  int n = 0;
  double tot = 0.0;
  for (auto& r : g_recs) {
    if (!r.closed || r.name != name) continue;
    if (hipEventSynchronize(r.b) != hipSuccess) return RNNT_EHIP;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) return RNNT_EHIP;
    ++n;
    tot += ms;
  }
  *launches = n;
  *total_ms = tot;
  return RNNT_OK;
}

int rnnt_profile_names(char* buf, size_t cap) {
  if (!buf || cap == 0) return RNNT_EINVAL;
  std::lock_guard<std::mutex> lk(g_mu);
  std::vector<std::string> seen;
  std::string out;
  for (auto& r : g_recs) {
    bool dup = false;
    for (auto& s : seen) dup = dup || (s == r.name);
    if (dup) continue;
    seen.push_back(r.name);
    if (!out.empty()) out += ",";
    out += r.name;
  }
  strncpy(buf, out.c_str(), cap - 1);
  buf[cap - 1] = 0;
  return RNNT_OK;
}

}  // extern "C"
