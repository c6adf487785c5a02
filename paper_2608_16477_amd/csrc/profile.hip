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

// Clock-sampling counters, PALLAS_K_COUNT x [cycles, wall ticks, workgroups],
// allocated on the device that is current at the first enable.
unsigned long long* g_clk = nullptr;

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

unsigned long long* profile_clock_slot(int cls) {
  if (!profile_on(cls) || !g_clk) return nullptr;
  return g_clk + 3 * cls;
}

void profile_record(int cls, hipEvent_t begin, hipEvent_t end) {
  std::lock_guard<std::mutex> lk(g_mu);
  g_pending.push_back({cls, begin, end});
}

}  // namespace pallas

extern "C" {

void pallas_profile_enable(uint32_t class_mask) {
  using namespace pallas;
  {
    std::lock_guard<std::mutex> lk(g_mu);
    if (class_mask && !g_clk) {
      void* p = nullptr;
      if (hipMalloc(&p, 3 * PALLAS_K_COUNT * sizeof(unsigned long long)) == hipSuccess &&
          hipMemset(p, 0, 3 * PALLAS_K_COUNT * sizeof(unsigned long long)) == hipSuccess)
        g_clk = static_cast<unsigned long long*>(p);
    }
  }
  g_mask.store(class_mask);
}

int pallas_profile_clock(int32_t kernel_class, double* mean_ghz, int64_t* workgroups) {
  using namespace pallas;
  if (kernel_class < 0 || kernel_class >= PALLAS_K_COUNT || !mean_ghz) return PALLAS_ERR_INVALID_ARG;
  *mean_ghz = 0.0;
  if (workgroups) *workgroups = 0;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_clk) return PALLAS_OK;
  unsigned long long v[3];
  int dev = 0, khz = 0;
  if (hipDeviceSynchronize() != hipSuccess ||
      hipMemcpy(v, g_clk + 3 * kernel_class, sizeof v, hipMemcpyDeviceToHost) != hipSuccess ||
      hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess)
    return PALLAS_ERR_HIP;
  if (v[1] > 0 && khz > 0) *mean_ghz = double(v[0]) / (double(v[1]) / (khz * 1e3)) / 1e9;
  if (workgroups) *workgroups = static_cast<int64_t>(v[2]);
  return PALLAS_OK;
}

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
  if (g_clk) (void)hipMemset(g_clk, 0, 3 * PALLAS_K_COUNT * sizeof(unsigned long long));
}

}  // extern "C"
