// SDMA copy-engine driver (see sdma.hpp).
#include "sdma.hpp"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <numeric>

namespace csg {

std::string hsa_error(hsa_status_t s) {
  const char* m = nullptr;
  if (hsa_status_string(s, &m) != HSA_STATUS_SUCCESS || !m) return "HSA status " + std::to_string(static_cast<int>(s));
  return m;
}

namespace {
struct AgentQuery {
  uint32_t bdf;
  uint32_t domain;
  hsa_agent_t found;
  bool ok;
};

hsa_status_t match_agent(hsa_agent_t a, void* data) {
  AgentQuery* q = static_cast<AgentQuery*>(data);
  hsa_device_type_t t;
  if (hsa_agent_get_info(a, HSA_AGENT_INFO_DEVICE, &t) != HSA_STATUS_SUCCESS || t != HSA_DEVICE_TYPE_GPU)
    return HSA_STATUS_SUCCESS;
  uint32_t bdf = 0, domain = 0;
  if (hsa_agent_get_info(a, static_cast<hsa_agent_info_t>(HSA_AMD_AGENT_INFO_BDFID), &bdf) != HSA_STATUS_SUCCESS)
    return HSA_STATUS_SUCCESS;
  (void)hsa_agent_get_info(a, static_cast<hsa_agent_info_t>(HSA_AMD_AGENT_INFO_DOMAIN), &domain);
  // compare bus and device; the function number is not reported by HIP
  if ((bdf >> 3) == (q->bdf >> 3) && domain == q->domain && !q->ok) {
    q->found = a;
    q->ok = true;
  }
  return HSA_STATUS_SUCCESS;
}
}  // namespace

std::string SdmaEngines::open(int hip_device, int max_engines, void* scratch_dst, const void* scratch_src) {
  close();
  int bus = 0, dev = 0, domain = 0;
  if (hipDeviceGetAttribute(&bus, hipDeviceAttributePciBusId, hip_device) != hipSuccess ||
      hipDeviceGetAttribute(&dev, hipDeviceAttributePciDeviceId, hip_device) != hipSuccess ||
      hipDeviceGetAttribute(&domain, hipDeviceAttributePciDomainId, hip_device) != hipSuccess)
    return "cannot read the device's PCI location";
  hsa_status_t s = hsa_init();  // reference counted; the HIP runtime already holds one
  if (s != HSA_STATUS_SUCCESS) return "hsa_init: " + hsa_error(s);
  hsa_inited_ = true;
  AgentQuery q{(static_cast<uint32_t>(bus) << 8) | (static_cast<uint32_t>(dev) << 3), static_cast<uint32_t>(domain),
               {0}, false};
  s = hsa_iterate_agents(match_agent, &q);
  if (s != HSA_STATUS_SUCCESS || !q.ok) {
    close();
    return "no HSA agent matches the HIP device";
  }
  agent_ = q.found;
  // Engines the runtime reports free for device-to-device copies. In a process whose
  // HIP runtime has already moved data the query can fail; then every engine id but
  // the first two (which the HIP runtime's own copies use first) is a candidate, and
  // each candidate is kept only if a warm-up copy on it completes.
  uint32_t mask = 0;
  s = hsa_amd_memory_copy_engine_status(agent_, agent_, &mask);
  if (s != HSA_STATUS_SUCCESS || mask == 0) mask = 0xfffcu;
  std::vector<hsa_amd_sdma_engine_id_t> candidates;
  for (int b = 0; b < 16; ++b)
    if (mask & (1u << b)) candidates.push_back(static_cast<hsa_amd_sdma_engine_id_t>(1u << b));
  // the first copy on an engine also pays its set-up cost; take it now
  for (hsa_amd_sdma_engine_id_t id : candidates) {
    if (max_engines > 0 && static_cast<int>(engines_.size()) >= max_engines) break;
    hsa_signal_t done;
    s = hsa_signal_create(1, 0, nullptr, &done);
    if (s != HSA_STATUS_SUCCESS) {
      close();
      return "hsa_signal_create: " + hsa_error(s);
    }
    s = hsa_amd_memory_async_copy_on_engine(scratch_dst, agent_, scratch_src, agent_, 4, 0, nullptr, done, id,
                                            /*force_copy_on_sdma=*/true);
    const hsa_signal_value_t left = (s == HSA_STATUS_SUCCESS) ? sdma_wait(done, 0, 2000) : 1;
    if (s != HSA_STATUS_SUCCESS || left == 0) hsa_signal_destroy(done);  // else the engine may still write it
    if (s == HSA_STATUS_SUCCESS && left == 0) engines_.push_back(id);
  }
  if (engines_.empty()) {
    close();
    return "no SDMA engine completed a device-to-device copy";
  }
  free_at_.assign(engines_.size(), std::chrono::steady_clock::time_point{});
  opened_ = true;
  return "";
}

void SdmaEngines::close() {
  engines_.clear();
  free_at_.clear();
  opened_ = false;
  if (hsa_inited_) {
    (void)hsa_shut_down();
    hsa_inited_ = false;
  }
}

hsa_status_t SdmaEngines::copy(void* dst, const void* src, size_t bytes, int engine, const hsa_signal_t* dep,
                               hsa_signal_t done) const {
  const hsa_amd_sdma_engine_id_t id = engines_[static_cast<size_t>(engine) % engines_.size()];
  return hsa_amd_memory_async_copy_on_engine(dst, agent_, src, agent_, bytes, dep ? 1u : 0u, dep, done, id,
                                             /*force_copy_on_sdma=*/true);
}

hsa_status_t SdmaEngines::copy_pieces(void* dst, const void* src, size_t bytes, int max_pieces, hsa_signal_t done,
                                      int budget_ms, int* pieces) {
  using Clock = std::chrono::steady_clock;
  const int n = count();
  const Clock::time_point now = Clock::now();
  auto start_us = [&](int e) {
    return std::chrono::duration<double, std::micro>(std::max(now, free_at_[static_cast<size_t>(e)]) - now).count();
  };
  std::vector<int> order(static_cast<size_t>(n));
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int x, int y) { return start_us(x) < start_us(y); });
  const int pmax = static_cast<int>(std::max<size_t>(
      1, std::min<size_t>({static_cast<size_t>(std::max(max_pieces, 1)), static_cast<size_t>(n), bytes / kMinPieceBytes})));
  // P pieces on the P engines free first land when the last of those engines is
  // through its share
  int best = 1;
  double best_us = start_us(order[0]) + static_cast<double>(bytes) / kEngineBytesPerUs;
  for (int q = 2; q <= pmax; ++q) {
    const double t = start_us(order[static_cast<size_t>(q - 1)]) + static_cast<double>(bytes) / q / kEngineBytesPerUs;
    if (t <= best_us - kPieceGainUs) {
      best = q;
      best_us = t;
    }
  }
  *pieces = best;
  if (best > 1) hsa_signal_add_relaxed(done, best - 1);
  // piece k covers [k * step, (k + 1) * step), the last one the rest; 64 KiB multiples
  const size_t step = (bytes / static_cast<size_t>(best)) & ~size_t{65535};
  for (int k = 0; k < best; ++k) {
    const size_t off = static_cast<size_t>(k) * step;
    const size_t len = k + 1 < best ? step : bytes - off;
    const int e = order[static_cast<size_t>(k)];
    const hsa_status_t s = copy(static_cast<char*>(dst) + off, static_cast<const char*>(src) + off, len, e, nullptr,
                                done);
    if (s != HSA_STATUS_SUCCESS) {
      // the k pieces issued bring `done` down to best - k; then no piece is in flight
      (void)sdma_wait(done, best - k, budget_ms);
      hsa_signal_subtract_relaxed(done, best - k - 1);
      return s;
    }
    free_at_[static_cast<size_t>(e)] =
        std::max(now, free_at_[static_cast<size_t>(e)]) +
        std::chrono::nanoseconds(static_cast<int64_t>(static_cast<double>(len) / kEngineBytesPerUs * 1000.0));
  }
  return HSA_STATUS_SUCCESS;
}

hsa_signal_value_t sdma_wait(hsa_signal_t s, hsa_signal_value_t value, int budget_ms) {
  const auto t0 = std::chrono::steady_clock::now();
  const auto budget = std::chrono::milliseconds(budget_ms);
  for (;;) {
    const hsa_signal_value_t v = hsa_signal_load_scacquire(s);
    if (v == value || v < 0) return v;
    if (std::chrono::steady_clock::now() - t0 > budget) return v;
  }
}

}  // namespace csg
