// SDMA copy-engine driver: device-to-device copies issued straight to chosen SDMA
// engines through the HSA runtime (hsa_amd_memory_async_copy_on_engine), with HSA
// signals for completion and for ordering one copy after another.
//
// Copies issued here never occupy a compute unit and never enter a HIP stream, so
// they progress while a persistent kernel holds every CU and polls the flags they
// raise. Spreading consecutive chunks over all engines multiplies the copy
// bandwidth (one engine moves about 48 GB/s device-to-device on MI355X).
#pragma once

#include <hsa/hsa.h>
#include <hsa/hsa_ext_amd.h>

#include <chrono>
#include <cstddef>
#include <string>
#include <vector>

namespace csg {

class SdmaEngines {
 public:
  SdmaEngines() = default;
  SdmaEngines(const SdmaEngines&) = delete;
  SdmaEngines& operator=(const SdmaEngines&) = delete;
  ~SdmaEngines() { close(); }

  // Finds the HSA agent of HIP device `hip_device` (by PCI location), lists the SDMA
  // engines usable for its device-to-device copies and keeps at most `max_engines`
  // (0 = all). Every engine is warmed up with one small copy. "" on success.
  std::string open(int hip_device, int max_engines, void* scratch_dst, const void* scratch_src);
  void close();

  int count() const { return static_cast<int>(engines_.size()); }
  // Completion signal for copies, consumed by GPU agents only: the runtime makes it
  // without an interrupt event (which costs the engines several microseconds per
  // copy), and its value may be read by kernels through signal_value_ptr. The calling
  // thread polls the value too.
  hsa_status_t make_signal(hsa_signal_value_t initial, hsa_signal_t* out) const {
    return hsa_amd_signal_create(initial, 0, nullptr, HSA_AMD_SIGNAL_AMD_GPU_ONLY, out);
  }
  // Address of a signal's value, for kernels to poll.
  static hsa_status_t signal_value_ptr(hsa_signal_t s, const int64_t** out) {
    volatile hsa_signal_value_t* vp = nullptr;
    const hsa_status_t st = hsa_amd_signal_value_pointer(s, &vp);
    *out = const_cast<const int64_t*>(reinterpret_cast<volatile int64_t*>(vp));
    return st;
  }
  bool is_open() const { return opened_; }

  // Copy `bytes` from src to dst on engine `engine % count()`. The copy starts once
  // `dep` (if non-null) reads 0 and decrements `done` when it has completed.
  hsa_status_t copy(void* dst, const void* src, size_t bytes, int engine, const hsa_signal_t* dep,
                    hsa_signal_t done) const;

  // Copy `bytes` from src to dst in up to `max_pieces` pieces of at least kMinPieceBytes,
  // each on its own engine. The engines are chosen by a model of their queues: each
  // engine works through the pieces given to it in order at kEngineBytesPerUs, so it
  // is expected to be free at a known time. The pieces go to the engines expected to
  // be free first, and their number is the one that lands the copy soonest; one piece
  // more is taken only when it brings the landing forward by at least kPieceGainUs. So
  // a copy issued while most engines are busy stays whole, and one issued while
  // engines are idle is spread over them.
  // `done` must read 1 for this copy when it is called: it is raised by pieces - 1
  // before the pieces are issued, and each piece decrements it, so it reads 0 once
  // every piece has landed. If issuing a piece fails, the call waits (at most
  // budget_ms) for the pieces already issued, sets `done` back to 1 and returns the
  // error: the state of a copy that was never issued. *pieces is the number chosen.
  hsa_status_t copy_pieces(void* dst, const void* src, size_t bytes, int max_pieces, hsa_signal_t done,
                           int budget_ms, int* pieces);

  static constexpr size_t kMinPieceBytes = size_t{512} << 10;
  static constexpr double kEngineBytesPerUs = 48000.0;  // about 48 GB/s per engine
  static constexpr double kPieceGainUs = 2.0;

 private:
  bool opened_ = false;
  bool hsa_inited_ = false;
  hsa_agent_t agent_{0};
  std::vector<hsa_amd_sdma_engine_id_t> engines_;
  std::vector<std::chrono::steady_clock::time_point> free_at_;  // copy_pieces' model, per engine
};

// Polls `s` until it reads `value` or `budget_ms` pass. Returns the last value read.
hsa_signal_value_t sdma_wait(hsa_signal_t s, hsa_signal_value_t value, int budget_ms);

std::string hsa_error(hsa_status_t s);

}  // namespace csg
