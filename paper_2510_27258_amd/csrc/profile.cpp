// Optional per-kernel timing for benchmarks.  While enabled, each kernel the
// C ABI launches is bracketed by two HIP events: the kernel's dispatch
// records its own start and end time into them (hipExtLaunchKernel), so the
// figure is the kernel's execution time without the gaps of the stream.  A
// bracket holding more than one launch (or a launch not made through
// prof_take) falls back to events recorded on the stream around it.
// hla_profile_summary() reads them back once the caller has synchronised.
#include <cstdio>
#include <cstring>
#include <map>
#include <string>
#include <vector>

#include "../../include/hla.h"
#include "profile.h"

namespace {
struct Rec {
  const char* name;
  int slot;
};
bool g_on = false;
std::vector<hipEvent_t> g_ev;   // 2 per record
std::vector<Rec> g_rec;
int g_cap = 0;
int g_open = -1;
int g_launches = 0;   // launches made inside the open bracket
}  // namespace

namespace hla {
void prof_start(const char* name, hipStream_t s) {
  if (!g_on || (int)g_rec.size() >= g_cap) { g_open = -1; return; }
  const int slot = (int)g_rec.size();
  g_rec.push_back({name, slot});
  (void)hipEventRecord(g_ev[2 * slot], s);
  g_open = slot;
  g_launches = 0;
}
void prof_stop(hipStream_t s) {
  if (!g_on || g_open < 0) return;
  if (g_launches != 1) (void)hipEventRecord(g_ev[2 * g_open + 1], s);
  g_open = -1;
}
bool prof_take(hipEvent_t* start, hipEvent_t* stop) {
  if (!g_on || g_open < 0) return false;
  if (++g_launches != 1) return false;
  *start = g_ev[2 * g_open];
  *stop = g_ev[2 * g_open + 1];
  return true;
}
hipError_t prof_launch(const void* fn, dim3 grid, dim3 block, void** args, size_t lds, hipStream_t s) {
  hipEvent_t e0, e1;
  if (prof_take(&e0, &e1)) return hipExtLaunchKernel(fn, grid, block, args, lds, s, e0, e1, 0);
  return hipLaunchKernel(fn, grid, block, args, lds, s);
}
}  // namespace hla

extern "C" {

int hla_profile_begin(int max_records) {
  if (max_records < 1) return HLA_ERR_INVALID;
  for (hipEvent_t e : g_ev) (void)hipEventDestroy(e);
  g_ev.assign(2 * (size_t)max_records, nullptr);
  for (auto& e : g_ev)
    if (hipEventCreate(&e) != hipSuccess) return HLA_ERR_HIP;
  g_rec.clear();
  g_cap = max_records;
  g_on = true;
  return HLA_OK;
}

int hla_profile_end(void) {
  g_on = false;
  return HLA_OK;
}

int hla_profile_summary(char* buf, size_t len) {
  std::map<std::string, std::pair<int, double>> acc;
  std::vector<std::string> order;
  for (const Rec& r : g_rec) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, g_ev[2 * r.slot], g_ev[2 * r.slot + 1]) != hipSuccess) return HLA_ERR_HIP;
    if (!acc.count(r.name)) order.push_back(r.name);
    acc[r.name].first += 1;
    acc[r.name].second += ms;
  }
  std::string out;
  char line[256];
  for (const auto& n : order) {
    snprintf(line, sizeof(line), "%s %d %.6f\n", n.c_str(), acc[n].first, acc[n].second);
    out += line;
  }
  if (!buf || len == 0) return HLA_ERR_INVALID;
  strncpy(buf, out.c_str(), len - 1);
  buf[len - 1] = '\0';
  g_rec.clear();
  return HLA_OK;
}

}  // extern "C"
