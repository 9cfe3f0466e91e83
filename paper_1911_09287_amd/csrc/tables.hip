// Small device tables owned by a plan (chirps and filter spectra of the 1-D
// transforms, roots of unity of the filter DFT, inverse-DFT weights of the
// weight gradient).  Each is built on
// the host in double precision and uploaded by the plan's first call that
// needs it on a device; the plan frees them when it is destroyed.
#include <cstring>
#include <mutex>
#include <new>
#include <utility>
#include <vector>

#include "common.hpp"

namespace blc {
namespace {

struct TabEntry {
  int dev;
  std::vector<long> key;
  float2* d;
};
std::mutex g_tab_mu;

}  // namespace

bl_status_t plan_table(const bl_conv_plan_s* p, const std::vector<long>& key,
                       const std::function<void(std::vector<float2>&)>& build, const float2** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return BL_ERR_HIP;
  std::lock_guard<std::mutex> lk(g_tab_mu);
  if (!p->tables) p->tables = new (std::nothrow) std::vector<TabEntry>();
  auto* cache = static_cast<std::vector<TabEntry>*>(p->tables);
  if (!cache) return BL_ERR_OOM;
  for (const TabEntry& e : *cache)
    if (e.dev == dev && e.key == key) {
      *out = e.d;
      return BL_OK;
    }
  std::vector<float2> host;
  build(host);
  float2* d = nullptr;
  if (hipMalloc(&d, host.size() * sizeof(float2)) != hipSuccess) return BL_ERR_OOM;
  if (hipMemcpy(d, host.data(), host.size() * sizeof(float2), hipMemcpyHostToDevice) != hipSuccess) {
    (void)hipFree(d);
    return BL_ERR_HIP;
  }
  cache->push_back(TabEntry{dev, key, d});
  *out = d;
  return BL_OK;
}

bl_status_t lds_opt_in(const void* kern, int bytes) {
  static std::mutex mu;
  static std::vector<std::pair<const void*, int>> done;  // (kernel, device)
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return BL_ERR_HIP;
  std::lock_guard<std::mutex> lk(mu);
  for (const auto& e : done)
    if (e.first == kern && e.second == dev) return BL_OK;
  if (hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, bytes) != hipSuccess) return BL_ERR_HIP;
  done.emplace_back(kern, dev);
  return BL_OK;
}

int device_cus() {
  static int count[64];  // per device; written once with the same value
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (count[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    count[dev] = n;
  }
  return count[dev];
}

long float_key(float x) {
  unsigned u;
  std::memcpy(&u, &x, sizeof u);
  return (long)u;
}

}  // namespace blc

void bl_plan_tables_free(void* tables) {
  if (!tables) return;
  auto* c = static_cast<std::vector<blc::TabEntry>*>(tables);
  int cur = 0;
  const bool have = hipGetDevice(&cur) == hipSuccess;
  for (const blc::TabEntry& e : *c)
    if (hipSetDevice(e.dev) == hipSuccess) (void)hipFree(e.d);
  if (have) (void)hipSetDevice(cur);
  delete c;
}
