// Process-wide per-kernel-class timing with HIP events.
#include <atomic>
#include <mutex>
#include <vector>

#include "profile.h"

namespace pallas {

namespace {

struct Pending {
  int cls;
  hipEvent_t begin, end;
};

std::atomic<uint32_t> g_mask{0};
std::mutex g_mu;
std::vector<Pending> g_pending;
std::vector<hipEvent_t> g_free;
double g_ms[PALLAS_K_COUNT];
int64_t g_launches[PALLAS_K_COUNT];

void release(hipEvent_t e) { g_free.push_back(e); }

}  // namespace

bool profile_on(int cls) { return (g_mask.load(std::memory_order_relaxed) >> cls) & 1u; }

hipEvent_t profile_event() {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_free.empty()) {
    hipEvent_t e = g_free.back();
    g_free.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void profile_record(int cls, hipEvent_t begin, hipEvent_t end) {
  std::lock_guard<std::mutex> lk(g_mu);
  g_pending.push_back({cls, begin, end});
}

}  // namespace pallas

extern "C" {

void pallas_profile_enable(uint32_t class_mask) { pallas::g_mask.store(class_mask); }

int pallas_profile_read(double* ms, int64_t* launches) {
  using namespace pallas;
  std::lock_guard<std::mutex> lk(g_mu);
  int rc = PALLAS_OK;
  for (const Pending& p : g_pending) {
    float t = 0.f;
    if (hipEventSynchronize(p.end) != hipSuccess || hipEventElapsedTime(&t, p.begin, p.end) != hipSuccess)
      rc = PALLAS_ERR_HIP;
    else if (p.cls >= 0 && p.cls < PALLAS_K_COUNT) {
      g_ms[p.cls] += t;
      g_launches[p.cls] += 1;
    }
    release(p.begin);
    release(p.end);
  }
  g_pending.clear();
  for (int k = 0; k < PALLAS_K_COUNT; ++k) {
    if (ms) ms[k] = g_ms[k];
    if (launches) launches[k] = g_launches[k];
  }
  return rc;
}

void pallas_profile_reset(void) {
  using namespace pallas;
  std::lock_guard<std::mutex> lk(g_mu);
  for (const Pending& p : g_pending) {
    (void)hipEventSynchronize(p.end);
    release(p.begin);
    release(p.end);
  }
  g_pending.clear();
  for (int k = 0; k < PALLAS_K_COUNT; ++k) {
    g_ms[k] = 0.0;
    g_launches[k] = 0;
  }
}

}  // extern "C"
