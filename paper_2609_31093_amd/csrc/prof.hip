// Opt-in per-kernel timing: when enabled, every internal kernel launch is
// bracketed by two hipEvents recorded on the launch stream; a report call
// waits for the events and returns per-kernel totals.  Disabled by default,
// in which case ProfScope does nothing.
#include <hip/hip_runtime.h>
#include <stdio.h>
#include <string.h>

#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/pisa.h"
#include "kernels.h"

namespace pisa {

namespace {
struct Rec {
  const char* name;
  hipEvent_t a, b;
};
std::mutex g_mu;
bool g_on = false;
std::vector<Rec> g_pending;
std::vector<hipEvent_t> g_free;
struct Acc {
  double ms = 0;
  long n = 0;
};
std::map<std::string, Acc> g_acc;

hipEvent_t get_event() {
  if (!g_free.empty()) {
    hipEvent_t e = g_free.back();
    g_free.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void drain_locked() {
  for (Rec& r : g_pending) {
    float ms = 0.f;
    if (r.a && r.b && hipEventSynchronize(r.b) == hipSuccess && hipEventElapsedTime(&ms, r.a, r.b) == hipSuccess) {
      Acc& acc = g_acc[r.name];
      acc.ms += ms;
      acc.n += 1;
    }
    if (r.a) g_free.push_back(r.a);
    if (r.b) g_free.push_back(r.b);
  }
  g_pending.clear();
}
}  // namespace

ProfScope::ProfScope(const char* name, hipStream_t st) : name_(name), st_(st), a_(nullptr) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_on) return;
  a_ = get_event();
  if (a_) hipEventRecord(static_cast<hipEvent_t>(a_), st_);
}

ProfScope::~ProfScope() {
  if (!a_) return;
  std::lock_guard<std::mutex> lk(g_mu);
  hipEvent_t b = get_event();
  if (b) hipEventRecord(b, st_);
  g_pending.push_back({name_, static_cast<hipEvent_t>(a_), b});
  if (g_pending.size() > 4096) drain_locked();
}

}  // namespace pisa

extern "C" {

int pisa_profile_enable(int on) {
  std::lock_guard<std::mutex> lk(pisa::g_mu);
  pisa::g_on = on != 0;
  return PISA_OK;
}

int pisa_profile_report(char* buf, size_t cap) {
  std::lock_guard<std::mutex> lk(pisa::g_mu);
  pisa::drain_locked();
  std::string out;
  for (auto& kv : pisa::g_acc) {
    char line[256];
    snprintf(line, sizeof(line), "%s %ld %.6f\n", kv.first.c_str(), kv.second.n, kv.second.ms);
    out += line;
  }
  pisa::g_acc.clear();
  if (buf && cap) {
    const size_t n = out.size() < cap - 1 ? out.size() : cap - 1;
    memcpy(buf, out.data(), n);
    buf[n] = 0;
  }
  return static_cast<int>(out.size());
}

}  // extern "C"
