// C ABI of the chunk-scheduled GEMM library (declared in include/csg.h) and the
// host runtime behind it: plan state on the device, the copy-engine driver that
// moves chunks and raises their flags, and the kernel launches.
//
// Copy-engine realization (Section 5.2, realization (1): copy engine with
// global-memory signals). Every chunk copy goes straight to an SDMA engine through
// the HSA runtime (sdma.cpp), consecutive chunks on consecutive engines, or, with
// copy_split, cut into pieces on the engines expected to be free first. A chunk's
// ready flag is the completion signal of its copy: a GPU-only HSA signal whose value
// the host sets to 1 before the call's kernel is launched and the engine brings to 0
// when the copy has landed (each piece of a cut copy brings it down by one, from the
// number of pieces); the kernel polls that value in memory. Signals come in
// two sets used by alternate calls, so a kernel still finishing the previous call
// never sees its signals reset. No copy enters a HIP stream: on this platform a
// stream wait (and the stream write/wait-value operations, which run as kernels)
// can end up behind the persistent kernel in a shared hardware queue, and a copy
// behind it could not progress until the kernel that waits for its flag ends.
//
// The ordering the copies need is enforced by the calling thread before it issues
// them (the caller's copy stream has reached the call; the earlier kernel that read
// the rows being rewritten has finished reading them). An overlap GEMM call returns
// once its copies are issued: its kernel waits for each chunk's copy, and
// csg_plan_check for all of them. Ring-attention and copy-only calls return once
// their copies have completed. This matches the paper's copy-engine backend, whose
// transfers are launched from the host (Section 2.3). Reduce-scatter output chunks
// are copied out by the calling thread as their completion flags (coherent host
// memory) rise; those copies complete after the call returns, and the next call's
// kernel waits for each before rewriting its rows.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <atomic>
#include <chrono>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <thread>
#include <vector>

#include "csg.h"
#include "attn.hpp"
#include "exec_tables.hpp"
#include "noalloc.hpp"
#include "kernels.hpp"
#include "planner.hpp"
#include "sdma.hpp"

namespace {

thread_local std::string g_last_error;

csg_status fail(csg_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

csg_status hip_fail(hipError_t e, const char* what) {
  return fail(e == hipErrorOutOfMemory ? CSG_ERR_NOMEM : CSG_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define CSG_HIP(expr)                                      \
  do {                                                     \
    hipError_t e_ = (expr);                                \
    if (e_ != hipSuccess) return hip_fail(e_, #expr);      \
  } while (0)

// Restores the caller's current device on scope exit.
struct DeviceGuard {
  int prev = -1;
  hipError_t err = hipSuccess;
  explicit DeviceGuard(int dev) {
    err = hipGetDevice(&prev);
    if (err == hipSuccess && prev != dev) err = hipSetDevice(dev);
  }
  ~DeviceGuard() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
};

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Epochs run 1 .. kEpochWrap - 1; on reaching it the emitted-flag words are cleared.
constexpr uint32_t kEpochWrap = 1u << 30;
constexpr int kTimingRing = 256;  // kernel launches whose durations a plan keeps
constexpr int64_t kCopySlab = 256 << 10;  // bytes per copy item of the copy workgroups
constexpr int32_t kDefaultCopyWorkgroups = 16;

}  // namespace

struct csg_schedule {
  csg::Schedule s;
};

struct csg_plan {
  csg_op op = CSG_AG_GEMM;
  bool attn = false;                   // a ring-attention plan (csg_attn_plan_create); op is unused
  int64_t M = 0, N = 0, K = 0;
  csg_dtype in_dtype = CSG_BF16, out_dtype = CSG_BF16;
  csg::Schedule sched;
  std::vector<int64_t> group_rows;
  csg_plan_cfg cfg{};
  csg::TileMap map;
  int device = -1;
  csg::KernelKey key{};
  int32_t grid = 0;
  std::vector<int32_t> remote_order;   // non-local chunk ids in arrival / emission order
  std::vector<float> delays_us;        // per remote chunk, in remote_order order
  uint32_t epoch = 0;
  bool kernel_pending[2] = {false, false};  // a kernel was launched with epoch parity i

  // device state
  csg::TileDesc* d_tiles = nullptr;
  int32_t* d_list_ptr = nullptr;
  int32_t* d_list_ids = nullptr;
  int32_t* d_raster = nullptr;
  int32_t* d_need = nullptr;
  int32_t* d_list_begin = nullptr;     // [kXcdLists + 1] per-die sub-list bounds (in units)
  float* d_ws = nullptr;               // split-K partial sums
  uint32_t* d_slot_count = nullptr;    // split-K finished slices per tile, [2][n_tiles]
  int32_t ws_slices = 0;               // partial-sum buffers of split tiles (0: nothing is split)
  int32_t tail_begin = 0;              // static dispatch: first unit dealt from the shared ticket
  uint64_t* d_trace = nullptr;         // per-unit trace words (cfg.trace)
  std::vector<csg::TileDesc> units;    // host copy of the execution list
  std::vector<int32_t> unit_raster;    // raster id per execution position
  bool lines_aligned = false;          // every chunk of A starts on a 128-byte line
  int32_t n_units = 0;                 // entries of the execution list
  const int64_t** d_ready[2] = {nullptr, nullptr};  // per signal set: [n_chunks] ready-value pointers
  int64_t* d_zero = nullptr;           // the "ready" value local chunks point at
  // per-call state, two sets by call parity (see GemmArgs::next_ticket)
  uint32_t* d_counters = nullptr;      // [2][n_chunks]
  uint32_t* d_ticket = nullptr;        // [2][kXcdLists]
  csg::DeviceDiag* d_diag = nullptr;   // [2]
  uint32_t reset_for_epoch = 0;        // call whose state set a launched kernel clears (0: none)
  uint32_t* h_out_flags = nullptr;     // coherent host memory, per chunk: the producer's emitted
                                       // flags; consumers: the call whose kernel has finished reading
                                       // the chunk's rows
  uint32_t last_kernel_epoch = 0;      // call number of the latest kernel launched (0: none)
  hipStream_t last_compute = nullptr;  // compute stream of the latest call (valid if has_last_compute)
  bool has_last_compute = false;
  // Consumer landing buffers recently read by this plan's kernels: the latest reader's
  // call number per distinct range (newest last), and the newest reader among ranges
  // dropped from the list. Copies into a range wait only for kernels that read it.
  struct LandingUse {
    uintptr_t base;
    size_t bytes;
    uint32_t epoch;
  };
  std::vector<LandingUse> landing_uses;
  uint32_t landing_dropped = 0;
  uint32_t* h_out_flags_dev = nullptr; // its device address
  uint32_t* d_scratch = nullptr;       // target of the engines' warm-up copies
  // csg_plan_join: per signal set, the value pointers of every copy signal of the set
  // (copies in, copies out, sends, partials), and the join kernel's timeout word
  const int64_t** d_join[2] = {nullptr, nullptr};
  int32_t n_join[2] = {0, 0};
  uint32_t* d_join_flag = nullptr;
  csg::SdmaEngines sdma;
  // Completion signals of the chunk copies, per set (calls alternate sets), per remote
  // chunk position: consumers' copies in, the producer's copies out.
  std::vector<hsa_signal_t> sig_ready[2];
  // GEMM + all-reduce, per set: sig_ready holds every chunk's last copy (emission
  // order); sig_send the reduce-scatter send of a non-local chunk, which the copy-in of
  // its reduced rows waits for; sig_part the landing of each other rank's partial sums
  // of an own chunk ([peer * own chunks + q]), polled by the own-shard tiles
  std::vector<hsa_signal_t> sig_send[2];
  std::vector<hsa_signal_t> sig_part[2];
  const int64_t** d_part_ready[2] = {nullptr, nullptr};
  int64_t ar_own_row0 = 0, ar_own_rows = 0;  // the own shard
  int32_t ar_chunk_rows = 0, ar_peers = 0, ar_own_shard = 0;
  // ring attention: heads, key/value heads, query rows; device arrays
  int32_t at_heads = 0, at_kv_heads = 0, at_q_rows = 0;
  int32_t* d_arrival = nullptr;        // [n_chunks] chunk id at each arrival position
  int32_t* d_chunk_rows = nullptr;     // [2 * n_chunks] key row begin / end by chunk id
  const void* ar_partials = nullptr;  // this call's partials landing buffer
  bool copies_in_flight = false;       // a call returned before its copies completed (consumers:
                                       // error paths only; producer: every call)
  int copies_set = 0;                  // signal set of those copies
  hipEvent_t ev_copy_in = nullptr;     // the caller's copy stream reached the call
  hipEvent_t ev_prologue = nullptr;    // the latest prologue finished
  bool prologue_queued = false;        // ev_prologue has been recorded
  hipEvent_t ev_kernel_done[2] = {nullptr, nullptr};  // by epoch parity
  hipEvent_t ev_k0[kTimingRing] = {};  // timing events around each kernel launch (ring)
  hipEvent_t ev_k1[kTimingRing] = {};
  uint64_t n_launches = 0;
  hipStream_t aux = nullptr;           // plan-internal transfers (diagnostics)
  csg_diag host_diag{};                // host-side wait failures of the last call
  uint32_t expected_units = 0;         // work units the last kernel launch had to run

  // Chunks moved by the kernel itself (cfg.copy_backend == CSG_COPY_KERNEL)
  csg::CopyItem* d_copy_items = nullptr;  // consumers: staging -> landing; producer: C -> outgoing
  int32_t n_copy_items = 0;
  int32_t* d_copy_chunk = nullptr;     // per remote position: chunk id
  int32_t* d_copy_parts = nullptr;     // per remote position: copy items
  uint32_t* d_copy_done = nullptr;     // per remote position: items finished
  int64_t* d_kready = nullptr;         // per chunk: ready word the copy workgroups clear
  const int64_t** d_ready_k = nullptr; // per chunk: its ready word (local chunks: d_zero)
  int32_t* d_chunk_sent = nullptr;     // per chunk: 1 if sent (producer)
  csg::CopyState* d_copy_state = nullptr;
  uint64_t* d_release_ticks = nullptr; // per remote position: cumulative release time, 100 MHz ticks
  bool release_set = false;

  int32_t n_chunks() const { return static_cast<int32_t>(sched.chunks.size()); }
  int32_t copy_workgroups() const { return cfg.copy_workgroups; }
  size_t n_flags() const { return static_cast<size_t>(std::max(n_chunks(), 1)); }
  uint32_t* counters(int set) const { return d_counters + set * n_flags(); }
  uint32_t* ticket(int set) const { return d_ticket + set * csg::kXcdLists; }
  csg::DeviceDiag* diag(int set) const { return d_diag + set; }
  uint32_t* slot_count(int set) const { return d_slot_count ? d_slot_count + set * map.n_tiles() : nullptr; }
  bool consumer() const { return op == CSG_AG_GEMM || op == CSG_GROUPED_GEMM || attention(); }
  bool attention() const { return attn; }
  // ring attention: copies per chunk (keys and values), both completing its signal
  hsa_signal_value_t copies_per_chunk() const { return attention() ? 2 : 1; }
  bool allreduce() const { return op == CSG_GEMM_AR; }
  // chunks that get copies, in the order the copies are issued: consumers and GEMM-RS,
  // the remote chunks; GEMM-AR, every chunk (own chunks are sent once reduced)
  const std::vector<int32_t>& copied_chunks() const { return allreduce() ? sched.order : remote_order; }
  bool kernel_copies() const { return cfg.copy_backend == CSG_COPY_KERNEL; }
};

namespace {

void free_plan_device(csg_plan* p) {
  if (p->device < 0) return;
  DeviceGuard g(p->device);
  // The plan's kernels poll its signals' values and read its device tables: wait for
  // them first (their waits are bounded, so they end), then for copies still in flight,
  // and only then destroy the signals and free the memory.
  for (hipEvent_t e : {p->ev_prologue, p->ev_kernel_done[0], p->ev_kernel_done[1]})
    if (e) (void)hipEventSynchronize(e);
  for (auto* sets : {p->sig_ready, p->sig_send, p->sig_part})
    for (int k = 0; k < 2; ++k)
      for (hsa_signal_t sgn : sets[k])
        if (sgn.handle) (void)csg::sdma_wait(sgn, 0, 10000);  // a copy may still be in flight
  for (auto* sets : {p->sig_ready, p->sig_send, p->sig_part})
    for (int k = 0; k < 2; ++k)
      for (hsa_signal_t sgn : sets[k])
        if (sgn.handle) hsa_signal_destroy(sgn);
  p->sdma.close();
  for (void* ptr : {static_cast<void*>(p->d_tiles), static_cast<void*>(p->d_list_ptr),
                    static_cast<void*>(p->d_list_ids), static_cast<void*>(p->d_raster), static_cast<void*>(p->d_need),
                    static_cast<void*>(p->d_list_begin), static_cast<void*>(p->d_ws),
                    static_cast<void*>(p->d_slot_count), static_cast<void*>(p->d_trace),
                    static_cast<void*>(p->d_ready[0]), static_cast<void*>(p->d_ready[1]),
                    static_cast<void*>(p->d_part_ready[0]), static_cast<void*>(p->d_part_ready[1]),
                    static_cast<void*>(p->d_zero),
                    static_cast<void*>(p->d_counters), static_cast<void*>(p->d_ticket), static_cast<void*>(p->d_diag),
                    static_cast<void*>(p->d_scratch), static_cast<void*>(p->d_copy_items),
                    static_cast<void*>(p->d_copy_chunk), static_cast<void*>(p->d_copy_parts),
                    static_cast<void*>(p->d_copy_done), static_cast<void*>(p->d_kready),
                    static_cast<void*>(p->d_ready_k), static_cast<void*>(p->d_chunk_sent),
                    static_cast<void*>(p->d_copy_state), static_cast<void*>(p->d_release_ticks),
                    static_cast<void*>(p->d_arrival), static_cast<void*>(p->d_chunk_rows),
                    static_cast<void*>(p->d_join[0]), static_cast<void*>(p->d_join[1]),
                    static_cast<void*>(p->d_join_flag)})
    if (ptr) (void)hipFree(ptr);
  if (p->h_out_flags) (void)hipHostFree(p->h_out_flags);
  for (hipEvent_t e : {p->ev_copy_in, p->ev_prologue, p->ev_kernel_done[0], p->ev_kernel_done[1]})
    if (e) (void)hipEventDestroy(e);
  for (int i = 0; i < kTimingRing; ++i) {
    if (p->ev_k0[i]) (void)hipEventDestroy(p->ev_k0[i]);
    if (p->ev_k1[i]) (void)hipEventDestroy(p->ev_k1[i]);
  }
  if (p->aux) (void)hipStreamDestroy(p->aux);
}

template <class T>
csg_status upload(T** dst, const std::vector<T>& src) {
  const size_t bytes = std::max<size_t>(src.size(), 1) * sizeof(T);
  CSG_HIP(hipMalloc(reinterpret_cast<void**>(dst), bytes));
  if (!src.empty()) CSG_HIP(hipMemcpy(*dst, src.data(), src.size() * sizeof(T), hipMemcpyHostToDevice));
  return CSG_OK;
}

int64_t in_bytes(const csg_plan* p) { return p->in_dtype == CSG_BF16 ? 2 : 4; }
int64_t out_bytes(const csg_plan* p) { return p->out_dtype == CSG_BF16 ? 2 : 4; }

// The join tables of csg_plan_join: per signal set, the completion values of every copy
// signal the set holds.
csg_status setup_join(csg_plan* p) {
  for (int set = 0; set < 2; ++set) {
    std::vector<const int64_t*> ptrs;
    for (auto* sets : {p->sig_ready, p->sig_send, p->sig_part})
      for (hsa_signal_t sgn : sets[set]) {
        const int64_t* vp = nullptr;
        const hsa_status_t hs = p->sdma.signal_value_ptr(sgn, &vp);
        if (hs != HSA_STATUS_SUCCESS) return fail(CSG_ERR_HIP, "copy signal: %s", csg::hsa_error(hs).c_str());
        ptrs.push_back(vp);
      }
    p->n_join[set] = static_cast<int32_t>(ptrs.size());
    const csg_status st = upload(&p->d_join[set], ptrs);
    if (st != CSG_OK) return st;
  }
  CSG_HIP(hipMalloc(&p->d_join_flag, 4));
  CSG_HIP(hipMemset(p->d_join_flag, 0, 4));
  return CSG_OK;
}

csg_status setup_device(csg_plan* p) {
  DeviceGuard g(p->device);
  if (g.err != hipSuccess) return hip_fail(g.err, "hipSetDevice");
  const csg::TileMap& m = p->map;
  const int32_t n_tiles = m.n_tiles();
  csg::ExecOptions eo;
  eo.consumer = p->consumer();
  eo.K = p->K;
  eo.in_bytes = in_bytes(p);
  eo.bk = p->cfg.bk;
  eo.split_k = p->cfg.split_k;
  eo.tail_split = p->cfg.tail_split;
  eo.tail_chunks = p->cfg.tail_chunks;
  eo.tail_taper = p->cfg.tail_taper;
  eo.tile_dispatch = p->cfg.tile_dispatch;
  eo.grid = p->grid;
  eo.tail_wave = p->cfg.tail_wave;
  csg::ExecTables et;
  csg::build_exec_tables(p->sched, m, eo, &et);
  const std::vector<csg::TileDesc>& tiles = et.units;
  const std::vector<int32_t>& lptr = et.list_ptr;
  const std::vector<int32_t>& lids = et.list_ids;
  const std::vector<int32_t>& raster = et.raster;
  const std::vector<int32_t>& need = et.need;
  const std::vector<int32_t>& list_begin = et.list_begin;
  const int32_t ws_slices = et.ws_slices;
  const int32_t n_units = static_cast<int32_t>(tiles.size());
  p->ws_slices = ws_slices;
  p->tail_begin = et.tail_begin;
  p->units = tiles;
  p->unit_raster = raster;
  p->n_units = n_units;
  p->lines_aligned = et.lines_aligned;
  csg_status st;
  if ((st = upload(&p->d_tiles, tiles)) != CSG_OK) return st;
  if ((st = upload(&p->d_list_ptr, lptr)) != CSG_OK) return st;
  if ((st = upload(&p->d_list_ids, lids)) != CSG_OK) return st;
  if ((st = upload(&p->d_raster, raster)) != CSG_OK) return st;
  if ((st = upload(&p->d_need, need)) != CSG_OK) return st;
  if ((st = upload(&p->d_list_begin, list_begin)) != CSG_OK) return st;
  const size_t nflag = static_cast<size_t>(std::max(p->n_chunks(), 1));
  CSG_HIP(hipMalloc(&p->d_zero, 64));
  CSG_HIP(hipMemset(p->d_zero, 0, 64));
  CSG_HIP(hipMalloc(&p->d_counters, 2 * nflag * 4));
  CSG_HIP(hipMemset(p->d_counters, 0, 2 * nflag * 4));
  CSG_HIP(hipMalloc(&p->d_ticket, 2 * csg::kXcdLists * 4));
  CSG_HIP(hipMemset(p->d_ticket, 0, 2 * csg::kXcdLists * 4));
  if (ws_slices > 0) {
    const size_t ws_bytes = static_cast<size_t>(ws_slices) * p->cfg.bm * p->cfg.bn * sizeof(float);
    CSG_HIP(hipMalloc(&p->d_ws, ws_bytes));
    CSG_HIP(hipMalloc(&p->d_slot_count, 2 * static_cast<size_t>(n_tiles) * 4));
    CSG_HIP(hipMemset(p->d_slot_count, 0, 2 * static_cast<size_t>(n_tiles) * 4));
  }
  if (p->cfg.trace) {
    const size_t words = static_cast<size_t>(std::max(n_units, 1)) * csg::kTraceWords;
    CSG_HIP(hipMalloc(&p->d_trace, words * sizeof(uint64_t)));
    CSG_HIP(hipMemset(p->d_trace, 0, words * sizeof(uint64_t)));
  }
  CSG_HIP(hipMalloc(&p->d_diag, 2 * sizeof(csg::DeviceDiag)));
  CSG_HIP(hipMemset(p->d_diag, 0, 2 * sizeof(csg::DeviceDiag)));
  CSG_HIP(hipHostMalloc(&p->h_out_flags, nflag * 4, hipHostMallocMapped | hipHostMallocCoherent));
  std::memset(p->h_out_flags, 0, nflag * 4);
  CSG_HIP(hipHostGetDevicePointer(reinterpret_cast<void**>(&p->h_out_flags_dev), p->h_out_flags, 0));
  CSG_HIP(hipMalloc(&p->d_scratch, 64));
  if (p->kernel_copies()) {
    // copy items: every remote chunk in arrival (emission) order, cut into slabs of
    // kCopySlab bytes; consumers move A rows staging -> landing, the producer (in
    // copy-only calls; its overlap calls send from the epilogue) C rows C -> outgoing
    const int64_t row_bytes = p->consumer() ? p->K * in_bytes(p) : p->N * out_bytes(p);
    std::vector<csg::CopyItem> items;
    std::vector<int32_t> parts, sent(p->n_chunks(), 0);
    std::vector<const int64_t*> words(p->n_chunks(), p->d_zero);
    // polled by workgroups on every die and written by others: fine-grained
    // (coherent) device memory
    CSG_HIP(hipExtMallocWithFlags(reinterpret_cast<void**>(&p->d_kready), nflag * 8, hipDeviceMallocFinegrained));
    CSG_HIP(hipMemset(p->d_kready, 0, nflag * 8));
    csg::build_copy_items(p->sched, p->remote_order, row_bytes, kCopySlab, &items, &parts);
    for (const int32_t cid : p->remote_order) {
      sent[cid] = 1;
      words[cid] = p->d_kready + cid;
    }
    p->n_copy_items = static_cast<int32_t>(items.size());
    if ((st = upload(&p->d_copy_items, items)) != CSG_OK) return st;
    if ((st = upload(&p->d_copy_chunk, p->remote_order)) != CSG_OK) return st;
    if ((st = upload(&p->d_copy_parts, parts)) != CSG_OK) return st;
    if ((st = upload(&p->d_chunk_sent, sent)) != CSG_OK) return st;
    if ((st = upload(&p->d_ready_k, words)) != CSG_OK) return st;
    const size_t n_remote = std::max<size_t>(p->remote_order.size(), 1);
    CSG_HIP(hipMalloc(&p->d_copy_done, n_remote * 4));
    CSG_HIP(hipMalloc(&p->d_release_ticks, n_remote * 8));
    CSG_HIP(hipMalloc(&p->d_copy_state, sizeof(csg::CopyState)));
    CSG_HIP(hipMemset(p->d_copy_state, 0, sizeof(csg::CopyState)));
  }
  CSG_HIP(hipDeviceSynchronize());
  std::string err = p->sdma.open(p->device, p->cfg.copy_engines, p->d_scratch, p->d_scratch + 8);
  if (!err.empty()) return fail(CSG_ERR_HIP, "copy engines: %s", err.c_str());
  const std::vector<int32_t>& copied = p->copied_chunks();
  const size_t n_copied = copied.size();
  auto make_set = [&](std::vector<hsa_signal_t>& sigs, size_t n, std::vector<const int64_t*>* ptrs,
                      const std::vector<int32_t>* slot) -> csg_status {
    sigs.assign(n, hsa_signal_t{0});
    for (size_t i = 0; i < n; ++i) {
      hsa_status_t hs = p->sdma.make_signal(0, &sigs[i]);
      const int64_t* vp = nullptr;
      if (hs == HSA_STATUS_SUCCESS) hs = p->sdma.signal_value_ptr(sigs[i], &vp);
      if (hs != HSA_STATUS_SUCCESS) return fail(CSG_ERR_NOMEM, "copy signal: %s", csg::hsa_error(hs).c_str());
      if (ptrs) (*ptrs)[slot ? (*slot)[i] : static_cast<int32_t>(i)] = vp;
    }
    return CSG_OK;
  };
  for (int set = 0; set < 2; ++set) {
    std::vector<const int64_t*> ptrs(p->n_chunks(), p->d_zero);  // chunks never copied: ready
    if ((st = make_set(p->sig_ready[set], n_copied, &ptrs, &copied)) != CSG_OK) return st;
    if ((st = upload(&p->d_ready[set], ptrs)) != CSG_OK) return st;
    if (p->allreduce()) {
      if ((st = make_set(p->sig_send[set], n_copied, nullptr, nullptr)) != CSG_OK) return st;
      const size_t n_part = static_cast<size_t>(p->ar_peers) * (p->ar_own_rows / p->ar_chunk_rows);
      std::vector<const int64_t*> pp(std::max<size_t>(n_part, 1), p->d_zero);
      if ((st = make_set(p->sig_part[set], n_part, &pp, nullptr)) != CSG_OK) return st;
      if ((st = upload(&p->d_part_ready[set], pp)) != CSG_OK) return st;
    }
  }
  CSG_HIP(hipEventCreateWithFlags(&p->ev_copy_in, hipEventDisableTiming));
  CSG_HIP(hipEventCreateWithFlags(&p->ev_prologue, hipEventDisableTiming));
  for (hipEvent_t& e : p->ev_kernel_done) CSG_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
  for (int i = 0; i < kTimingRing; ++i) {
    CSG_HIP(hipEventCreate(&p->ev_k0[i]));
    CSG_HIP(hipEventCreate(&p->ev_k1[i]));
  }
  CSG_HIP(hipStreamCreateWithFlags(&p->aux, hipStreamNonBlocking));
  if ((st = setup_join(p)) != CSG_OK) return st;
  CSG_HIP(hipDeviceSynchronize());
  return CSG_OK;
}


using Clock = std::chrono::steady_clock;

void spin_until(Clock::time_point t) {
  while (Clock::now() < t) {
  }
}

// Host-side wait for an event, bounded; polls so the caller resumes within microseconds.
csg_status host_wait(csg_plan* p, hipEvent_t e, const char* what) {
  const Clock::time_point t0 = Clock::now();
  const auto budget = std::chrono::milliseconds(p->cfg.timeout_ms) * 4;
  for (;;) {
    const hipError_t q = hipEventQuery(e);
    if (q == hipSuccess) return CSG_OK;
    if (q != hipErrorNotReady) return hip_fail(q, what);
    if (Clock::now() - t0 > budget) {
      p->host_diag = csg_diag{1, -1, -1, 0, p->epoch, 0};
      return fail(CSG_ERR_TIMEOUT, "%s did not complete in time", what);
    }
  }
}

struct CallState {
  int prev_parity = 0;
  bool prev_kernel = false;
  bool wrapped = false;  // the call number restarted: every earlier kernel has finished
};

// The signals this call's copies complete: one set per call parity.
std::vector<hsa_signal_t>& call_signals(csg_plan* p) { return p->sig_ready[p->epoch & 1]; }

// Waits for copies a previous call left running: a consumer's after an error return
// (before its signals are armed again); with `all`, also the producer's copy-outs,
// which complete after their call returns.
csg_status drain_copies(csg_plan* p, bool all) {
  if (!p->copies_in_flight || (!all && !p->consumer())) return CSG_OK;
  const int budget = p->cfg.timeout_ms * 4;
  for (auto* sets : {p->sig_ready, p->sig_send, p->sig_part})
    for (int set = 0; set < 2; ++set)
      for (hsa_signal_t sgn : sets[set])
        if (csg::sdma_wait(sgn, 0, budget) > 0)
          return fail(CSG_ERR_TIMEOUT, "copies of an earlier call did not complete");
  p->copies_in_flight = false;
  return CSG_OK;
}

// Front half of a call: the call number advances and the call's ready signals are
// armed.
csg_status begin_call(csg_plan* p, csg_mode mode, CallState* cs) {
  if (mode != CSG_MODE_OVERLAP && mode != CSG_MODE_COMPUTE_ONLY && mode != CSG_MODE_COPY_ONLY)
    return fail(CSG_ERR_INVALID, "unknown mode %d", static_cast<int>(mode));
  csg_status st = drain_copies(p, false);
  if (st != CSG_OK) return st;
  cs->prev_parity = p->epoch & 1;
  cs->prev_kernel = p->kernel_pending[cs->prev_parity];
  if (p->epoch + 1 >= kEpochWrap) {
    // the producer's emitted flags hold epochs: once no kernel can still write one,
    // clear them and restart at 2 (so the new epoch's parity differs from the last one's)
    for (int par = 0; par < 2; ++par)
      if (p->kernel_pending[par] && (st = host_wait(p, p->ev_kernel_done[par], "an earlier kernel")) != CSG_OK)
        return st;
    std::memset(p->h_out_flags, 0, static_cast<size_t>(std::max(p->n_chunks(), 1)) * 4);
    p->epoch = 1;
    // every earlier kernel has finished: no copy of this call waits for one
    p->landing_uses.clear();
    p->landing_dropped = 0;
    cs->wrapped = true;
  }
  ++p->epoch;
  p->host_diag = csg_diag{0, -1, -1, 0, p->epoch, 0};
  // the signals this call's kernel polls: consumers', the copies in of their chunks;
  // GEMM + all-reduce, the landing of the other ranks' partial sums
  const int set = p->epoch & 1;
  std::vector<hsa_signal_t>* polled = nullptr;
  if (p->consumer() && !p->remote_order.empty() && !p->kernel_copies()) polled = &p->sig_ready[set];
  if (p->allreduce() && !p->sig_part[set].empty()) polled = &p->sig_part[set];
  if (polled) {
    // this call's signal set was last polled by the kernel two calls back, which must
    // be done before the set is armed again (it normally ended long ago)
    if (p->kernel_pending[set] && (st = host_wait(p, p->ev_kernel_done[set], "the kernel two calls back")) != CSG_OK)
      return st;
    // the partials' copies complete after their call returns (a copy-only call has no
    // kernel that waited for them): each must be done before its signal is armed again
    if (p->allreduce())
      for (hsa_signal_t sgn : *polled)
        if (csg::sdma_wait(sgn, 0, p->cfg.timeout_ms * 4) != 0)
          return fail(CSG_ERR_TIMEOUT, "an earlier copy of a partial sum did not complete");
    // compute-only: every chunk ready; otherwise one decrement per copy of the chunk
    const hsa_signal_value_t v = mode == CSG_MODE_COMPUTE_ONLY ? 0 : p->copies_per_chunk();
    for (hsa_signal_t sgn : *polled) hsa_signal_store_relaxed(sgn, v);
    std::atomic_thread_fence(std::memory_order_seq_cst);  // armed before the kernel launch below
  }
  p->kernel_pending[p->epoch & 1] = false;
  return CSG_OK;
}

// The call's prologue on the compute stream (before its kernel, if any).
// The previous call's kernel cleared this call's state set when it ran, unless the
// previous call launched none (copy-only, an error) or the copies are the kernel's own
// (their ready words depend on this call's mode): then the prologue kernel does.
csg_status launch_prologue_call(csg_plan* p, csg_mode mode, hipStream_t compute) {
  // The per-call state sets and the copies' write-after-read waits rely on the plan's
  // kernels and prologues running in call order. A call on another compute stream than
  // the previous one therefore first waits, on the device, for the latest kernel and the
  // latest prologue queued on the earlier streams (a copy-only call queues a prologue
  // that clears a state set, and no kernel).
  if (p->has_last_compute && p->last_compute != compute) {
    if (p->last_kernel_epoch) CSG_HIP(hipStreamWaitEvent(compute, p->ev_kernel_done[p->last_kernel_epoch & 1], 0));
    if (p->prologue_queued) CSG_HIP(hipStreamWaitEvent(compute, p->ev_prologue, 0));
  }
  p->last_compute = compute;
  p->has_last_compute = true;
  const int set = p->epoch & 1;
  if (mode != CSG_MODE_COPY_ONLY && !p->kernel_copies() && p->reset_for_epoch == p->epoch) return CSG_OK;
  csg::PrologueArgs pa{};
  pa.counters = p->counters(set);
  pa.n_chunks = p->n_chunks();
  pa.epoch = p->epoch;
  pa.ticket = p->ticket(set);
  pa.diag = p->diag(set);
  pa.slot_count = p->slot_count(set);
  pa.n_slots = p->ws_slices > 0 ? p->map.n_tiles() : 0;
  if (p->kernel_copies()) {
    // consumers' remote chunks are not there until the copy workgroups move them;
    // the producer waits for nothing before rewriting C (no copy out reads it later)
    pa.ready_words = p->d_kready;
    pa.ready_value = (p->consumer() && mode != CSG_MODE_COMPUTE_ONLY) ? 1 : 0;
    pa.copy_done = p->d_copy_done;
    pa.n_remote = static_cast<int32_t>(p->remote_order.size());
    pa.copy_state = p->d_copy_state;
  }
  CSG_HIP(csg::launch_prologue(pa, compute));
  CSG_HIP(hipEventRecord(p->ev_prologue, compute));
  p->prologue_queued = true;
  return CSG_OK;
}

// Ordering the copies need, enforced from the host (see the file comment).
csg_status ready_copies(csg_plan* p, hipStream_t copy, const CallState& cs, bool war_on_previous_kernel) {
  csg_status st = CSG_OK;
  const hipError_t q = hipStreamQuery(copy);  // idle: nothing to wait for
  if (q == hipErrorNotReady) {
    CSG_HIP(hipEventRecord(p->ev_copy_in, copy));
    if ((st = host_wait(p, p->ev_copy_in, "the copy stream's earlier work")) != CSG_OK) return st;
  } else if (q != hipSuccess) {
    return hip_fail(q, "hipStreamQuery");
  }
  if (war_on_previous_kernel && cs.prev_kernel) {
    st = host_wait(p, p->ev_kernel_done[cs.prev_parity], "the previous call's kernel");
    if (st != CSG_OK) return st;
  }
  p->copies_in_flight = true;
  p->copies_set = p->epoch & 1;
  return CSG_OK;
}

// Waits until every issued copy of this call has completed.
csg_status finish_copies(csg_plan* p, size_t issued) {
  const int budget = p->cfg.timeout_ms * 4;
  const std::vector<hsa_signal_t>& sigs = call_signals(p);
  for (size_t i = 0; i < issued; ++i) {
    hsa_signal_value_t v = csg::sdma_wait(sigs[i], 0, budget);
    if (v < 0) return fail(CSG_ERR_HIP, "SDMA copy %zu reported an error", i);
    if (v != 0) {
      p->host_diag = csg_diag{1, p->remote_order[i], -1, 0, p->epoch, 0};
      return fail(CSG_ERR_TIMEOUT, "SDMA copy of chunk %d did not complete in time", p->remote_order[i]);
    }
  }
  p->copies_in_flight = false;
  return CSG_OK;
}

// Chunk moves a kernel launch does itself (copy backend CSG_COPY_KERNEL).
struct KernelCopies {
  bool copy = false;              // copy workgroups move the copy items src -> dst
  const void* src = nullptr;
  void* dst = nullptr;
  void* c2 = nullptr;             // producer: the epilogue also stores sent chunks here
};

csg_status launch_gemm(csg_plan* p, const void* A, const void* B, void* C, csg_mode mode, hipStream_t compute,
                       const KernelCopies* kc = nullptr) {
  csg::GemmArgs a{};
  a.A = A;
  a.B = B;
  a.C = C;
  a.M = p->M;
  a.N = p->N;
  a.K = p->K;
  a.b_group_stride = p->op == CSG_GROUPED_GEMM ? p->N * p->K : 0;
  a.tiles = p->d_tiles;
  a.list_ptr = p->d_list_ptr;
  a.list_ids = p->d_list_ids;
  a.raster = p->d_raster;
  // consumers wait for this call's copies in; the producer, before overwriting a
  // chunk's rows of C, for the previous call's copy out of them
  a.ready = p->d_ready[p->consumer() ? (p->epoch & 1) : ((p->epoch + 1) & 1)];
  const int set = p->epoch & 1, next = set ^ 1;
  a.counters = p->counters(set);
  a.need = p->d_need;
  a.out_flags = p->h_out_flags_dev;
  a.ticket = p->ticket(set);
  a.list_begin = p->d_list_begin;
  a.diag = p->diag(set);
  a.timeout_ticks = static_cast<uint64_t>(p->cfg.timeout_ms) * 100000ull;  // 100 MHz wall clock
  a.epoch = p->epoch;
  a.n_tiles = p->n_units;
  a.ws = p->d_ws;
  a.slot_count = p->slot_count(set);
  if (!p->kernel_copies()) {
    // clear the next call's set in this kernel (the next call then needs no prologue)
    a.next_ticket = p->ticket(next);
    a.next_counters = p->counters(next);
    a.next_slot_count = p->slot_count(next);
    a.next_diag = p->diag(next);
    a.next_n_slots = p->ws_slices > 0 ? p->map.n_tiles() : 0;
  }
  a.n_chunks = p->n_chunks();
  a.dynamic_ticket = p->cfg.tile_dispatch == 2 ? 0 : 1;
  a.tail_begin = p->tail_begin;
  // Idle workgroups take other dies' units (split tiles exchange partial sums through
  // memory, so their slices may run on any die).
  a.steal = 1;
  a.trace = p->d_trace;
  // only copies of this call leave rows fresh in HBM; without them the warm-up loads
  // would only cost time
  a.n_tiles_n = (p->consumer() && mode == CSG_MODE_OVERLAP && p->cfg.warm_rows != 2) ? p->map.n_tiles_n : 0;
  a.acquire_fresh = (p->consumer() && (!p->lines_aligned || reinterpret_cast<uintptr_t>(A) % 128 != 0)) ? 1 : 0;
  int32_t grid = p->grid;
  if (kc) {
    // kernel-moved chunks have ready words of their own, which the prologue set
    a.ready = p->d_ready_k;
    if (mode == CSG_MODE_COPY_ONLY) {
      a.n_tiles = 0;  // the copy workgroups alone
      a.n_tiles_n = 0;
      grid = p->copy_workgroups();
    }
    if (kc->copy && p->n_copy_items > 0) {
      a.copy_items = p->d_copy_items;
      a.n_copy_items = p->n_copy_items;
      a.copy_wgs = p->copy_workgroups();
      a.copy_src = static_cast<const unsigned char*>(kc->src);
      a.copy_dst = static_cast<unsigned char*>(kc->dst);
      a.copy_chunk = p->d_copy_chunk;
      a.copy_parts = p->d_copy_parts;
      a.copy_done = p->d_copy_done;
      a.copy_ready = p->d_kready;
      a.copy_state = p->d_copy_state;
      a.release_ticks = p->release_set ? p->d_release_ticks : nullptr;
    }
    if (kc->c2) {
      a.C2 = kc->c2;
      a.chunk_sent = p->d_chunk_sent;
    }
  }
  if (p->allreduce()) {
    a.partials = static_cast<const unsigned char*>(p->ar_partials);
    a.partial_ready = p->d_part_ready[p->epoch & 1];
    a.own_row0 = p->ar_own_row0;
    a.own_rows = p->ar_own_rows;
    a.n_peers = p->ar_peers;
    a.own_chunk_rows = p->ar_chunk_rows;
    a.own_shard = p->ar_own_shard;
  }
  p->expected_units = static_cast<uint32_t>(a.n_tiles);
  const int slot = static_cast<int>(p->n_launches % kTimingRing);
  CSG_HIP(csg::launch_chunk_gemm(p->key, a, grid, compute, p->ev_k0[slot], p->ev_k1[slot]));
  p->reset_for_epoch = a.next_ticket ? p->epoch + 1 : 0;
  ++p->n_launches;
  CSG_HIP(hipEventRecord(p->ev_kernel_done[p->epoch & 1], compute));
  p->kernel_pending[p->epoch & 1] = true;
  p->last_kernel_epoch = p->epoch;
  return CSG_OK;
}

constexpr size_t kLandingHistory = 4;

// The kernel that copies into landing rows [base, base + bytes) have to wait for, and
// whether they may do so chunk by chunk. The newest kernel that read an overlapping range
// decides (the plan's kernels run in call order on one stream, so once it has started
// reading, every older kernel has finished): when it read exactly this range, a chunk's
// copy waits for that kernel to finish reading the chunk; when it read a different,
// overlapping range (or the range is unknown because the history dropped it), every
// copy waits until that kernel has finished reading all chunks. 0: no kernel to wait for.
uint32_t landing_reader(const csg_plan* p, const void* base, size_t bytes, bool* per_chunk) {
  const uintptr_t b = reinterpret_cast<uintptr_t>(base);
  uint32_t e = p->landing_dropped;
  *per_chunk = false;
  for (const csg_plan::LandingUse& u : p->landing_uses) {
    const bool overlap = u.base < b + bytes && b < u.base + u.bytes;
    if (overlap && u.epoch > e) {
      e = u.epoch;
      *per_chunk = u.base == b && u.bytes == bytes;
    }
  }
  return e;
}

// Records that this call's kernel (p->epoch) reads landing rows [base, base + bytes).
void note_landing_reader(csg_plan* p, const void* base, size_t bytes) {
  const uintptr_t b = reinterpret_cast<uintptr_t>(base);
  auto& uses = p->landing_uses;
  for (size_t i = 0; i < uses.size(); ++i)
    if (uses[i].base == b && uses[i].bytes == bytes) {
      uses.erase(uses.begin() + static_cast<std::ptrdiff_t>(i));
      break;
    }
  uses.push_back({b, bytes, p->epoch});
  if (uses.size() > kLandingHistory) {
    p->landing_dropped = std::max(p->landing_dropped, uses.front().epoch);
    uses.erase(uses.begin());
  }
}

// Consumer copies: staging -> landing per remote chunk, on engine (i mod engines)
// for the i-th remote chunk in arrival order; each completes the chunk's (armed)
// ready signal. Before overwriting a chunk's rows the issuer waits until the kernel
// that read them last (call prev_reader) is done with them: that kernel reports it per
// chunk (its consumed words), and its completion event settles it for every chunk
// (also when it gave up early). With all_chunks the first copy waits until that kernel
// has finished reading every chunk (it read an overlapping but different range). Copy
// delays release chunk i at the sum of the first i delays after the call started.
struct CopyIssuer {
  csg_plan* p;
  void* landing;
  const void* staging;
  uint32_t prev_reader;
  Clock::time_point t0;
  size_t next = 0;
  double release_us = 0.0;
  bool prev_done;
  void* landing2 = nullptr;        // ring attention: values (landing / staging: keys)
  const void* staging2 = nullptr;
  bool all_chunks = false;

  CopyIssuer(csg_plan* plan, void* l, const void* s, uint32_t prev)
      : p(plan), landing(l), staging(s), prev_reader(prev), t0(Clock::now()), prev_done(prev == 0) {}

  // Waits until kernel prev_reader has finished reading chunk cid (false with !block
  // when it has not yet).
  csg_status wait_read(int32_t cid, bool block, bool* ready) {
    const int prev_parity = static_cast<int>(prev_reader & 1);
    const auto budget = std::chrono::milliseconds(p->cfg.timeout_ms) * 4;
    const volatile uint32_t* f = p->h_out_flags + cid;
    const Clock::time_point tw = Clock::now();
    uint32_t spins = 0;
    *ready = true;
    while (!prev_done && *f < prev_reader) {
      if (!block) {
        *ready = false;
        return CSG_OK;
      }
      if ((++spins & 255u) == 0) {
        const hipError_t q = hipEventQuery(p->ev_kernel_done[prev_parity]);
        if (q == hipSuccess) {
          prev_done = true;
          break;
        }
        if (q != hipErrorNotReady) return hip_fail(q, "the previous call's kernel");
      }
      if (Clock::now() - tw > budget) {
        p->host_diag = csg_diag{1, cid, -1, *f, p->epoch, 0};
        return fail(CSG_ERR_TIMEOUT, "the previous kernel did not finish reading chunk %d in time", cid);
      }
    }
    return CSG_OK;
  }

  // Issues copies in arrival order. Without `block` it stops at the first copy that
  // would have to wait (for its release time or for the previous kernel).
  csg_status run(bool block) {
    const int64_t row_bytes = p->attention() ? int64_t{p->at_kv_heads} * csg::kAttnHeadDim * 2 : p->K * in_bytes(p);
    const std::vector<hsa_signal_t>& sigs = call_signals(p);
    if (all_chunks && !prev_done) {
      for (int32_t cid = 0; cid < p->n_chunks(); ++cid) {
        bool ready = true;
        const csg_status st = wait_read(cid, block, &ready);
        if (st != CSG_OK) {
          (void)finish_copies(p, next);
          return st;
        }
        if (!ready) return CSG_OK;
      }
      prev_done = true;
    }
    for (; next < p->remote_order.size(); ++next) {
      const size_t i = next;
      const int32_t cid = p->remote_order[i];
      const csg::ChunkDesc& c = p->sched.chunks[cid];
      if (!p->delays_us.empty()) {
        const Clock::time_point due =
            t0 + std::chrono::nanoseconds(static_cast<int64_t>((release_us + p->delays_us[i]) * 1000.0));
        if (!block && Clock::now() < due) return CSG_OK;
        spin_until(due);
      }
      if (!prev_done) {
        bool ready = true;
        const csg_status st = wait_read(cid, block, &ready);
        if (st != CSG_OK) {
          (void)finish_copies(p, i);
          return st;
        }
        if (!ready) return CSG_OK;
      }
      if (!p->delays_us.empty()) release_us += p->delays_us[i];
      const int64_t off = c.row_begin * row_bytes;
      const int64_t bytes = (c.row_end - c.row_begin) * row_bytes;
      const int eng = static_cast<int>(i % p->sdma.count());
      int pieces = 1;
      hsa_status_t hs =
          p->cfg.copy_split > 1
              ? p->sdma.copy_pieces(static_cast<char*>(landing) + off, static_cast<const char*>(staging) + off,
                                    static_cast<size_t>(bytes), p->cfg.copy_split, sigs[i], p->cfg.timeout_ms * 4,
                                    &pieces)
              : p->sdma.copy(static_cast<char*>(landing) + off, static_cast<const char*>(staging) + off,
                             static_cast<size_t>(bytes), eng, nullptr, sigs[i]);
      // ring attention: the values follow on the next engine; the chunk's signal,
      // armed to 2, reaches 0 when both copies have completed
      if (hs == HSA_STATUS_SUCCESS && landing2)
        hs = p->sdma.copy(static_cast<char*>(landing2) + off, static_cast<const char*>(staging2) + off,
                          static_cast<size_t>(bytes), eng + 1, nullptr, sigs[i]);
      if (hs != HSA_STATUS_SUCCESS) {
        // the chunks not copied keep their signals armed: the kernel's bounded waits for
        // them expire and it reports them through csg_plan_check
        (void)finish_copies(p, i);
        return fail(CSG_ERR_HIP, "SDMA copy of chunk %d: %s", cid, csg::hsa_error(hs).c_str());
      }
    }
    return CSG_OK;
  }
};

// Ring attention: device state of a plan (work units, chunk tables, per-call state,
// copy engines and the per-chunk signals of the key/value copies).
csg_status setup_attn_device(csg_plan* p) {
  DeviceGuard g(p->device);
  if (g.err != hipSuccess) return hip_fail(g.err, "hipSetDevice");
  p->n_units = ((p->at_q_rows + csg::kAttnBlockQ - 1) / csg::kAttnBlockQ) * p->at_heads;
  std::vector<int32_t> rows(2 * static_cast<size_t>(p->n_chunks()));
  for (int32_t c = 0; c < p->n_chunks(); ++c) {
    rows[2 * c] = static_cast<int32_t>(p->sched.chunks[c].row_begin);
    rows[2 * c + 1] = static_cast<int32_t>(p->sched.chunks[c].row_end);
  }
  csg_status st;
  if ((st = upload(&p->d_arrival, p->sched.order)) != CSG_OK) return st;
  if ((st = upload(&p->d_chunk_rows, rows)) != CSG_OK) return st;
  const size_t nflag = p->n_flags();
  CSG_HIP(hipMalloc(&p->d_zero, 64));
  CSG_HIP(hipMemset(p->d_zero, 0, 64));
  CSG_HIP(hipMalloc(&p->d_counters, 2 * nflag * 4));
  CSG_HIP(hipMemset(p->d_counters, 0, 2 * nflag * 4));
  CSG_HIP(hipMalloc(&p->d_ticket, 2 * csg::kXcdLists * 4));
  CSG_HIP(hipMemset(p->d_ticket, 0, 2 * csg::kXcdLists * 4));
  CSG_HIP(hipMalloc(&p->d_diag, 2 * sizeof(csg::DeviceDiag)));
  CSG_HIP(hipMemset(p->d_diag, 0, 2 * sizeof(csg::DeviceDiag)));
  CSG_HIP(hipHostMalloc(&p->h_out_flags, nflag * 4, hipHostMallocMapped | hipHostMallocCoherent));
  std::memset(p->h_out_flags, 0, nflag * 4);
  CSG_HIP(hipHostGetDevicePointer(reinterpret_cast<void**>(&p->h_out_flags_dev), p->h_out_flags, 0));
  CSG_HIP(hipMalloc(&p->d_scratch, 64));
  CSG_HIP(hipDeviceSynchronize());
  std::string err = p->sdma.open(p->device, p->cfg.copy_engines, p->d_scratch, p->d_scratch + 8);
  if (!err.empty()) return fail(CSG_ERR_HIP, "copy engines: %s", err.c_str());
  for (int set = 0; set < 2; ++set) {
    p->sig_ready[set].assign(p->remote_order.size(), hsa_signal_t{0});
    std::vector<const int64_t*> ptrs(p->n_chunks(), p->d_zero);  // local chunks: never copied
    for (size_t i = 0; i < p->remote_order.size(); ++i) {
      hsa_status_t hs = p->sdma.make_signal(0, &p->sig_ready[set][i]);
      const int64_t* vp = nullptr;
      if (hs == HSA_STATUS_SUCCESS) hs = p->sdma.signal_value_ptr(p->sig_ready[set][i], &vp);
      if (hs != HSA_STATUS_SUCCESS) return fail(CSG_ERR_NOMEM, "copy signal: %s", csg::hsa_error(hs).c_str());
      ptrs[p->remote_order[i]] = vp;
    }
    if ((st = upload(&p->d_ready[set], ptrs)) != CSG_OK) return st;
  }
  CSG_HIP(hipEventCreateWithFlags(&p->ev_copy_in, hipEventDisableTiming));
  CSG_HIP(hipEventCreateWithFlags(&p->ev_prologue, hipEventDisableTiming));
  for (hipEvent_t& e : p->ev_kernel_done) CSG_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));
  for (int i = 0; i < kTimingRing; ++i) {
    CSG_HIP(hipEventCreate(&p->ev_k0[i]));
    CSG_HIP(hipEventCreate(&p->ev_k1[i]));
  }
  CSG_HIP(hipStreamCreateWithFlags(&p->aux, hipStreamNonBlocking));
  if ((st = setup_join(p)) != CSG_OK) return st;
  CSG_HIP(hipDeviceSynchronize());
  return CSG_OK;
}

csg_status launch_attn(csg_plan* p, const void* q, const void* k, const void* v, void* o, void* lse,
                       hipStream_t compute) {
  const int set = p->epoch & 1, next = set ^ 1;
  csg::AttnArgs a{};
  a.Q = static_cast<const uint16_t*>(q);
  a.K = static_cast<const uint16_t*>(k);
  a.V = static_cast<const uint16_t*>(v);
  a.O = static_cast<uint16_t*>(o);
  a.LSE = static_cast<float*>(lse);
  a.Sq = p->at_q_rows;
  a.H = p->at_heads;
  a.Hkv = p->at_kv_heads;
  a.n_units = p->n_units;
  a.n_chunks = p->n_chunks();
  a.arrival = p->d_arrival;
  a.chunk_rows = p->d_chunk_rows;
  a.ready = p->d_ready[set];
  a.counters = p->counters(set);
  a.out_flags = p->h_out_flags_dev;
  a.ticket = p->ticket(set);
  a.diag = p->diag(set);
  a.timeout_ticks = static_cast<uint64_t>(p->cfg.timeout_ms) * 100000ull;  // 100 MHz wall clock
  a.epoch = p->epoch;
  a.scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt(static_cast<double>(csg::kAttnHeadDim)));
  a.next_ticket = p->ticket(next);
  a.next_counters = p->counters(next);
  a.next_diag = p->diag(next);
  const int slot = static_cast<int>(p->n_launches % kTimingRing);
  CSG_HIP(csg::launch_ring_attn(a, p->grid, compute, p->ev_k0[slot], p->ev_k1[slot]));
  p->reset_for_epoch = p->epoch + 1;
  p->expected_units = static_cast<uint32_t>(p->n_units);
  ++p->n_launches;
  CSG_HIP(hipEventRecord(p->ev_kernel_done[p->epoch & 1], compute));
  p->kernel_pending[p->epoch & 1] = true;
  p->last_kernel_epoch = p->epoch;
  return CSG_OK;
}

// A call whose chunks the kernel moves itself: the prologue and one kernel launch on
// the compute stream, nothing on the copy stream, no host waits. Consumers: the copy
// workgroups move staging -> landing (copy-only: they alone run). Producer: overlap
// calls send from the epilogue (c2 = outgoing); copy-only calls move C -> outgoing.
csg_status kernel_copy_call(csg_plan* p, const void* a, const void* staging, const void* b, void* c, void* outgoing,
                            csg_mode mode, hipStream_t compute) {
  CallState cs;
  csg_status st = begin_call(p, mode, &cs);
  if (st != CSG_OK) return st;
  if ((st = launch_prologue_call(p, mode, compute)) != CSG_OK) return st;
  KernelCopies kc;
  if (p->consumer()) {
    kc.copy = mode != CSG_MODE_COMPUTE_ONLY;
    kc.src = staging;
    kc.dst = const_cast<void*>(a);
  } else if (mode == CSG_MODE_COPY_ONLY) {
    kc.copy = true;
    kc.src = c;
    kc.dst = outgoing;
  } else if (mode == CSG_MODE_OVERLAP) {
    kc.c2 = outgoing;
  }
  return launch_gemm(p, a, b, c, mode, compute, &kc);
}

csg_status consumer_call(csg_plan* p, void* landing, const void* staging, const void* b, void* c, csg_mode mode,
                         void* compute_v, void* copy_v) {
  if (p->device < 0) return fail(CSG_ERR_STATE, "host-only plan (created with device < 0) cannot run");
  if (!landing || !b || !c || (mode != CSG_MODE_COMPUTE_ONLY && !staging && !p->remote_order.empty()))
    return fail(CSG_ERR_INVALID, "NULL buffer");
  if (!aligned16(landing) || !aligned16(staging) || !aligned16(b) || !aligned16(c))
    return fail(CSG_ERR_INVALID, "buffers must be 16-byte aligned");
  hipStream_t compute = static_cast<hipStream_t>(compute_v), copy = static_cast<hipStream_t>(copy_v);
  DeviceGuard g(p->device);
  if (g.err != hipSuccess) return hip_fail(g.err, "hipSetDevice");
  if (p->kernel_copies()) return kernel_copy_call(p, landing, staging, b, c, nullptr, mode, compute);
  CallState cs;
  // the kernel that last read these landing rows (before this call's own)
  const size_t landing_bytes = static_cast<size_t>(p->M) * static_cast<size_t>(p->K) * in_bytes(p);
  bool per_chunk = false;
  const uint32_t prev_reader = landing_reader(p, landing, landing_bytes, &per_chunk);
  csg_status st = begin_call(p, mode, &cs);
  if (st != CSG_OK) return st;
  const bool copies = mode != CSG_MODE_COMPUTE_ONLY && !p->remote_order.empty();
  CopyIssuer issuer(p, landing, staging, cs.wrapped ? 0u : prev_reader);
  issuer.all_chunks = !per_chunk;
  if (copies) {
    // the copies that need not wait go first (they take the longest to land), then the
    // kernel is queued: it starts as soon as the previous kernel ends and waits for its
    // chunks, while the host releases the remaining copies
    if ((st = ready_copies(p, copy, cs, false)) != CSG_OK) return st;
    if ((st = issuer.run(false)) != CSG_OK) return st;
  }
  if ((st = launch_prologue_call(p, mode, compute)) != CSG_OK) return st;
  if (mode != CSG_MODE_COPY_ONLY) {
    if ((st = launch_gemm(p, landing, b, c, mode, compute)) != CSG_OK) return st;
    note_landing_reader(p, landing, landing_bytes);
  }
  if (!copies) return CSG_OK;
  if ((st = issuer.run(true)) != CSG_OK) return st;
  if (mode == CSG_MODE_OVERLAP) {
    // Every copy is issued. This call's kernel waits for each of them (a chunk's tiles
    // wait for its signal), the signal set is armed again only after that kernel has
    // finished (two calls on), and a later copy into these landing rows waits for the
    // kernel to have read them: nothing needs the copies to have completed when the call
    // returns, and the engines move on to the next call's copies without a gap.
    p->copies_in_flight = false;
    return CSG_OK;
  }
  // Copy-only: the copies complete on their own. The next call waits for them before it
  // arms a signal again, csg_plan_check waits for them, and csg_plan_join makes a
  // stream wait for them on the device.
  return CSG_OK;
}

// ---- the allocation-free all-gather GEMM (csg_ag_gemm_noalloc) ----------------------
// Its tables and per-call words live in the library's static device scratch, at the
// fixed offsets below; nothing is allocated per call or per schedule.
constexpr int32_t kNaMaxChunks = 4096;   // also the kernels' ready-bitmap bound
constexpr int32_t kNaMaxUnits = 16384;   // tiles
constexpr int32_t kNaMaxNnz = 32768;     // (tile, remote chunk) pairs
constexpr int32_t kNaMaxItems = 16384;   // 256 KiB copy slabs: 4 GiB of remote rows

struct NaLayout {
  // per-call words, reset by the prologue of every call
  size_t diag, ticket, copy_state, counters, out_flags, kready, copy_done;
  // tables, written when a call's schedule or shape differs from the previous call's
  size_t tables, zero, tiles, list_ptr, list_ids, raster, list_begin, need, ready, items, copy_chunk, copy_parts;
  size_t end;
};

NaLayout na_layout() {
  NaLayout L{};
  size_t o = 0;
  auto take = [&o](size_t bytes) {
    const size_t at = o;
    o = (o + bytes + 255) & ~size_t{255};
    return at;
  };
  L.diag = take(sizeof(csg::DeviceDiag));
  L.ticket = take(csg::kXcdLists * 4);
  L.copy_state = take(sizeof(csg::CopyState));
  L.counters = take(kNaMaxChunks * 4);
  L.out_flags = take(kNaMaxChunks * 4);
  L.kready = take(kNaMaxChunks * 8);
  L.copy_done = take(kNaMaxChunks * 4);
  L.tables = o;
  L.zero = take(64);
  L.tiles = take(kNaMaxUnits * sizeof(csg::TileDesc));
  L.list_ptr = take((kNaMaxUnits + 1) * 4);
  L.list_ids = take(kNaMaxNnz * 4);
  L.raster = take(kNaMaxUnits * 4);
  L.list_begin = take((csg::kXcdLists + 1) * 4);
  L.need = take(kNaMaxChunks * 4);
  L.ready = take(kNaMaxChunks * 8);
  L.items = take(kNaMaxItems * sizeof(csg::CopyItem));
  L.copy_chunk = take(kNaMaxChunks * 4);
  L.copy_parts = take(kNaMaxChunks * 4);
  L.end = o;
  return L;
}

// What a device's scratch currently holds, and the host image of its tables.
struct NaDevice {
  bool checked = false;          // csg_device_check passed
  int32_t grid[4] = {0, 0, 0, 0};  // persistent grid per (input, output) dtype pair
  uint64_t sig = 0;              // signature of the tables in the scratch (0: none)
  std::vector<unsigned char> image;
  int32_t n_units = 0, n_remote = 0, n_items = 0, n_tiles_n = 0;
  bool lines_aligned = true;
  uint32_t calls = 0;
};
std::mutex g_na_mu;
NaDevice g_na[64];

uint64_t na_signature(const csg::Schedule& s, int64_t M, int64_t N, int64_t K, csg_dtype in, csg_dtype out) {
  uint64_t h = 1469598103934665603ull;
  auto mix = [&h](uint64_t v) {
    for (int i = 0; i < 8; ++i) {
      h ^= (v >> (8 * i)) & 0xffu;
      h *= 1099511628211ull;
    }
  };
  mix(static_cast<uint64_t>(M));
  mix(static_cast<uint64_t>(N));
  mix(static_cast<uint64_t>(K));
  mix(static_cast<uint64_t>(in) * 16 + static_cast<uint64_t>(out));
  for (const csg::ChunkDesc& c : s.chunks) {
    mix(static_cast<uint64_t>(c.row_begin));
    mix(static_cast<uint64_t>(c.row_end));
    mix(static_cast<uint64_t>(c.is_local));
  }
  for (int32_t o : s.order) mix(static_cast<uint64_t>(o));
  return h | 1u;  // never 0
}

}  // namespace

// =====================================================================================
// C ABI
// =====================================================================================
extern "C" {

const char* csg_version(void) { return "csg 0.1.0 (gfx950)"; }

const char* csg_status_str(csg_status s) {
  switch (s) {
    case CSG_OK: return "CSG_OK";
    case CSG_ERR_INVALID: return "CSG_ERR_INVALID";
    case CSG_ERR_UNSUPPORTED: return "CSG_ERR_UNSUPPORTED";
    case CSG_ERR_HIP: return "CSG_ERR_HIP";
    case CSG_ERR_NOMEM: return "CSG_ERR_NOMEM";
    case CSG_ERR_TIMEOUT: return "CSG_ERR_TIMEOUT";
    case CSG_ERR_STATE: return "CSG_ERR_STATE";
  }
  return "CSG_ERR_UNKNOWN";
}

const char* csg_last_error(void) { return g_last_error.c_str(); }

csg_status csg_device_check(int device, char* arch, size_t arch_len) {
  hipDeviceProp_t prop;
  hipError_t e = hipGetDeviceProperties(&prop, device);
  if (e != hipSuccess) return hip_fail(e, "hipGetDeviceProperties");
  if (arch && arch_len) {
    std::strncpy(arch, prop.gcnArchName, arch_len - 1);
    arch[arch_len - 1] = '\0';
  }
  if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
    return fail(CSG_ERR_UNSUPPORTED, "device %d is %s; this library is built for gfx950 only", device,
                prop.gcnArchName);
  return CSG_OK;
}

csg_status csg_schedule_create(const csg_chunk* chunks, int32_t n, const int32_t* order, csg_schedule** out) {
  if (!out) return fail(CSG_ERR_INVALID, "out is NULL");
  *out = nullptr;
  if (!chunks || !order || n < 1) return fail(CSG_ERR_INVALID, "chunks/order NULL or n < 1");
  csg::Schedule s;
  for (int32_t i = 0; i < n; ++i) {
    if (chunks[i].reserved != 0) return fail(CSG_ERR_INVALID, "chunk %d: reserved field must be 0", i);
    s.chunks.push_back({chunks[i].row_begin, chunks[i].row_end, chunks[i].src_rank, chunks[i].group,
                        chunks[i].is_local ? 1 : 0});
  }
  s.order.assign(order, order + n);
  std::string err = csg::validate_schedule(s.chunks, s.order);
  if (!err.empty()) return fail(CSG_ERR_INVALID, "%s", err.c_str());
  s.total_rows = s.chunks.back().row_end;
  csg_schedule* r = new (std::nothrow) csg_schedule{std::move(s)};
  if (!r) return fail(CSG_ERR_NOMEM, "out of host memory");
  *out = r;
  return CSG_OK;
}

csg_status csg_schedule_uniform(int32_t world, int32_t rank, int64_t shard_rows, int32_t chunks_per_shard,
                                csg_order order, const int32_t* remote_perm_host, csg_schedule** out) {
  if (!out) return fail(CSG_ERR_INVALID, "out is NULL");
  *out = nullptr;
  if (order < CSG_ORDER_RING || order > CSG_ORDER_RS_RING) return fail(CSG_ERR_INVALID, "unknown order");
  csg::Schedule s;
  std::string err = csg::make_uniform_schedule(world, rank, shard_rows, chunks_per_shard,
                                               static_cast<csg::OrderKind>(order), remote_perm_host, &s);
  if (!err.empty()) return fail(CSG_ERR_INVALID, "%s", err.c_str());
  csg_schedule* r = new (std::nothrow) csg_schedule{std::move(s)};
  if (!r) return fail(CSG_ERR_NOMEM, "out of host memory");
  *out = r;
  return CSG_OK;
}

csg_status csg_schedule_grouped(int32_t world, int32_t rank, int32_t n_groups, const int64_t* counts_host,
                                csg_schedule** out) {
  if (!out) return fail(CSG_ERR_INVALID, "out is NULL");
  *out = nullptr;
  csg::Schedule s;
  std::string err = csg::make_grouped_schedule(world, rank, n_groups, counts_host, &s);
  if (!err.empty()) return fail(CSG_ERR_INVALID, "%s", err.c_str());
  csg_schedule* r = new (std::nothrow) csg_schedule{std::move(s)};
  if (!r) return fail(CSG_ERR_NOMEM, "out of host memory");
  *out = r;
  return CSG_OK;
}

csg_status csg_schedule_info(const csg_schedule* s, int32_t* n_chunks, int64_t* total_rows) {
  if (!s) return fail(CSG_ERR_INVALID, "schedule is NULL");
  if (n_chunks) *n_chunks = static_cast<int32_t>(s->s.chunks.size());
  if (total_rows) *total_rows = s->s.total_rows;
  return CSG_OK;
}

csg_status csg_schedule_get(const csg_schedule* s, csg_chunk* chunks_host, int32_t* order_host) {
  if (!s) return fail(CSG_ERR_INVALID, "schedule is NULL");
  for (size_t i = 0; i < s->s.chunks.size(); ++i) {
    const csg::ChunkDesc& c = s->s.chunks[i];
    if (chunks_host) chunks_host[i] = csg_chunk{c.row_begin, c.row_end, c.src_rank, c.group, c.is_local, 0};
    if (order_host) order_host[i] = s->s.order[i];
  }
  return CSG_OK;
}

void csg_schedule_destroy(csg_schedule* s) { delete s; }

csg_status csg_plan_create(csg_op op, int64_t M, int64_t N, int64_t K, csg_dtype in_dtype, csg_dtype out_dtype,
                           const csg_schedule* s, const int64_t* group_rows_host, int32_t n_groups,
                           const csg_plan_cfg* cfg, int device, csg_plan** out) {
  if (!out) return fail(CSG_ERR_INVALID, "out is NULL");
  *out = nullptr;
  if (!s) return fail(CSG_ERR_INVALID, "schedule is NULL");
  if (op < CSG_AG_GEMM || op > CSG_GEMM_AR) return fail(CSG_ERR_INVALID, "unknown op");
  if ((in_dtype != CSG_BF16 && in_dtype != CSG_F32) || (out_dtype != CSG_BF16 && out_dtype != CSG_F32))
    return fail(CSG_ERR_INVALID, "unknown dtype");
  if (M < 1 || N < 1 || K < 1 || M > 0x7fffffff || N > 0x7fffffff || K > (1 << 22))
    return fail(CSG_ERR_INVALID, "shape out of range");
  std::vector<int64_t> groups;
  if (op == CSG_GROUPED_GEMM) {
    if (!group_rows_host || n_groups < 1) return fail(CSG_ERR_INVALID, "grouped GEMM needs group rows");
    groups.assign(group_rows_host, group_rows_host + n_groups);
  } else if (group_rows_host || n_groups) {
    return fail(CSG_ERR_INVALID, "group rows are only for the grouped GEMM");
  }
  csg_plan_cfg c = cfg ? *cfg : csg_plan_cfg{};
  const bool bf16 = in_dtype == CSG_BF16;
  if (c.bm == 0) c.bm = bf16 ? 256 : 64;
  if (c.bn == 0) c.bn = bf16 ? 256 : 64;
  if (c.bk == 0) c.bk = bf16 ? 64 : 16;
  if (c.timeout_ms == 0) c.timeout_ms = 2000;
  if (c.split_k == 0) c.split_k = 1;
  if (c.copy_workgroups == 0) c.copy_workgroups = kDefaultCopyWorkgroups;
  if (c.bm < 1 || c.bn < 1 || c.bk < 1 || c.copy_engines < 0 || c.copy_engines > 32 || c.timeout_ms < 1 ||
      c.split_k < 1 || c.split_k > 64 || c.tail_split < 0 || c.tail_split > 64 || c.tail_chunks < 0 ||
      c.trace < 0 || c.trace > 1 || c.warm_rows < 0 || c.warm_rows > 2 || c.copy_backend < 0 ||
      c.copy_backend > CSG_COPY_KERNEL || c.copy_workgroups < 0 || c.copy_workgroups > 4096 ||
      c.num_workgroups < 0 || c.tile_dispatch < 0 || c.tile_dispatch > 2 || c.intra_order < 0 ||
      c.intra_order > 1 || c.group_m < 0 || c.tail_wave < 0 || c.tail_wave > 64 || c.copy_split < 0 ||
      c.copy_split > 32 || c.tail_taper < 0 || c.tail_taper > 1)
    return fail(CSG_ERR_INVALID, "bad plan configuration");
  if (c.copy_split > 1 && (c.copy_backend != CSG_COPY_SDMA || op == CSG_GEMM_AR))
    return fail(CSG_ERR_UNSUPPORTED, "copy_split cuts the copy engines' chunk copies of all-gather, grouped and "
                                     "reduce-scatter plans");
  if (c.group_m == 0) c.group_m = 8;
  // split plans keep the grid a multiple of the die count (round-robin dispatch then
  // gives every die the same number of workgroups, and each die's list its share)
  if ((c.split_k > 1 || (c.tail_split > 1 && c.tail_chunks > 0) || c.tail_wave > 1) && c.tile_dispatch != 2 &&
      c.num_workgroups > 0 && c.num_workgroups % csg::kXcdLists != 0)
    return fail(CSG_ERR_INVALID, "with split tiles num_workgroups must be a multiple of %d", csg::kXcdLists);

  csg_plan* p = new (std::nothrow) csg_plan;
  if (!p) return fail(CSG_ERR_NOMEM, "out of host memory");
  p->op = op;
  p->M = M;
  p->N = N;
  p->K = K;
  p->in_dtype = in_dtype;
  p->out_dtype = out_dtype;
  p->sched = s->s;
  p->group_rows = groups;
  p->cfg = c;
  std::string err =
      csg::build_tile_map(p->sched, M, N, c.bm, c.bn, !p->consumer(), groups, &p->map, c.intra_order, c.group_m);
  if (!err.empty()) {
    delete p;
    return fail(CSG_ERR_INVALID, "%s", err.c_str());
  }
  for (int32_t c_id : p->sched.order)
    if (!p->sched.chunks[c_id].is_local) p->remote_order.push_back(c_id);
  if (op == CSG_GEMM_AR) {
    // the own shard: the local chunks, contiguous; every chunk the same height; tiles
    // never straddle the own shard's edges; no split tiles; copies by the engines
    const std::vector<csg::ChunkDesc>& ch = p->sched.chunks;
    const int64_t h = ch[0].row_end - ch[0].row_begin;
    int64_t own0 = -1, own1 = -1;
    std::string why;
    for (const csg::ChunkDesc& x : ch) {
      if (x.row_end - x.row_begin != h) why = "every chunk must have the same number of rows";
      if (x.is_local) {
        if (own0 < 0) own0 = x.row_begin;
        else if (x.row_begin != own1) why = "the local chunks must be contiguous (the own shard)";
        own1 = x.row_end;
      }
    }
    if (why.empty() && own0 < 0) why = "a GEMM + all-reduce plan needs local chunks (the own shard)";
    const int64_t S = own1 - own0;
    if (why.empty() && M % S != 0) why = "M must be a multiple of the own shard's rows";
    if (why.empty() && (own0 % c.bm != 0 || (own1 % c.bm != 0 && own1 != M)))
      why = "the own shard must start and end on a tile-row boundary (bm)";
    if (why.empty() && (c.split_k > 1 || (c.tail_split > 1 && c.tail_chunks > 0) || c.tail_wave > 1))
      why = "GEMM + all-reduce splits no tile";
    if (why.empty() && c.copy_backend != CSG_COPY_SDMA) why = "GEMM + all-reduce copies with the SDMA engines";
    if (!why.empty()) {
      delete p;
      return fail(CSG_ERR_UNSUPPORTED, "%s", why.c_str());
    }
    p->ar_own_row0 = own0;
    p->ar_own_rows = S;
    p->ar_chunk_rows = static_cast<int32_t>(h);
    p->ar_peers = static_cast<int32_t>(M / S - 1);
    p->ar_own_shard = static_cast<int32_t>(own0 / S);
  }
  if (op == CSG_GEMM_RS && c.copy_backend == CSG_COPY_KERNEL)
    for (const csg::ChunkDesc& ch : p->sched.chunks)
      if (ch.row_begin % c.bm != 0) {
        delete p;
        return fail(CSG_ERR_UNSUPPORTED,
                    "sending from the epilogue needs every chunk to start on a multiple of bm = %d (row %lld)", c.bm,
                    static_cast<long long>(ch.row_begin));
      }

  // every kernel variant keeps a per-workgroup bitmap of the chunks it has seen ready
  // (consumers: landed; producers: the previous call's copy out of the chunk done)
  if (p->n_chunks() > csg::kernel_max_chunks()) {
    delete p;
    return fail(CSG_ERR_UNSUPPORTED, "at most %d chunks", csg::kernel_max_chunks());
  }
  // the main loops step K by bk with no partial step, and the epilogue stores runs of
  // four columns (host-only plans too: they describe a plan a device would run)
  if (K % c.bk != 0 || N % 4 != 0) {
    delete p;
    return fail(CSG_ERR_UNSUPPORTED, "K must be a multiple of %d and N a multiple of 4", c.bk);
  }
  if (device >= 0) {
    p->key = csg::KernelKey{bf16 ? csg::InType::BF16 : csg::InType::F32, out_dtype == CSG_BF16, !p->consumer(),
                            c.bm, c.bn, c.bk, p->allreduce()};
    if (!csg::kernel_supported(p->key)) {
      delete p;
      return fail(CSG_ERR_UNSUPPORTED, "no kernel for dtype %d->%d tile %dx%dx%d", in_dtype, out_dtype, c.bm, c.bn,
                  c.bk);
    }
    // a tile's rows of A, B and C are addressed with 32-bit buffer offsets
    const int64_t ib = bf16 ? 2 : 4, ob = out_dtype == CSG_BF16 ? 2 : 4;
    if (static_cast<int64_t>(std::max(c.bm, c.bn)) * K * ib >= (int64_t{1} << 31) ||
        static_cast<int64_t>(c.bm) * N * ob >= (int64_t{1} << 30)) {
      delete p;
      return fail(CSG_ERR_UNSUPPORTED, "a %d-row tile of A/B (K = %lld) or of C (N = %lld) exceeds the 32-bit offset range",
                  std::max(c.bm, c.bn), static_cast<long long>(K), static_cast<long long>(N));
    }
    char arch[64];
    csg_status st = csg_device_check(device, arch, sizeof arch);
    if (st != CSG_OK) {
      delete p;
      return st;
    }
    p->device = device;
    {
      DeviceGuard g(device);
      hipError_t e = g.err != hipSuccess ? g.err : csg::kernel_grid(p->key, device, &p->grid);
      if (e != hipSuccess) {
        p->device = -1;
        delete p;
        return hip_fail(e, "occupancy query");
      }
    }
    if (c.num_workgroups > 0) p->grid = c.num_workgroups;
    st = setup_device(p);
    if (st != CSG_OK) {
      std::string msg = g_last_error;
      free_plan_device(p);
      delete p;
      g_last_error = msg;
      return st;
    }
  }
  *out = p;
  return CSG_OK;
}

csg_status csg_plan_info_get(const csg_plan* p, csg_plan_info* info) {
  if (!p || !info) return fail(CSG_ERR_INVALID, "NULL argument");
  info->n_tiles = p->map.n_tiles();
  info->n_chunks = p->n_chunks();
  info->nnz = static_cast<int32_t>(p->map.tile_chunks.size());
  info->n_tiles_n = p->map.n_tiles_n;
  info->num_workgroups = p->device >= 0 ? p->grid : 0;
  info->bm = p->cfg.bm;
  info->bn = p->cfg.bn;
  info->bk = p->cfg.bk;
  info->n_units = p->device >= 0 ? p->n_units : 0;
  return CSG_OK;
}

csg_status csg_plan_get_map(const csg_plan* p, int32_t* tile_ptr, int32_t* tile_chunks, int32_t* chunk_ptr,
                            int32_t* chunk_tiles, int32_t* tile_order) {
  if (!p) return fail(CSG_ERR_INVALID, "plan is NULL");
  const csg::TileMap& m = p->map;
  auto cp = [](int32_t* dst, const std::vector<int32_t>& v) {
    if (dst && !v.empty()) std::memcpy(dst, v.data(), v.size() * sizeof(int32_t));
  };
  cp(tile_ptr, m.tile_ptr);
  cp(tile_chunks, m.tile_chunks);
  cp(chunk_ptr, m.chunk_ptr);
  cp(chunk_tiles, m.chunk_tiles);
  cp(tile_order, m.order);
  return CSG_OK;
}

csg_status csg_plan_set_copy_delays(csg_plan* p, const float* delay_us_host, int32_t n) {
  if (!p) return fail(CSG_ERR_INVALID, "plan is NULL");
  if (!delay_us_host) {
    p->delays_us.clear();
    p->release_set = false;
    return CSG_OK;
  }
  if (n != static_cast<int32_t>(p->remote_order.size()))
    return fail(CSG_ERR_INVALID, "need %zu delays (one per remote chunk), got %d", p->remote_order.size(), n);
  for (int32_t i = 0; i < n; ++i)
    if (!(delay_us_host[i] >= 0.0f) || delay_us_host[i] > 1e6f) return fail(CSG_ERR_INVALID, "bad delay %d", i);
  p->delays_us.assign(delay_us_host, delay_us_host + n);
  if (p->device >= 0 && p->kernel_copies() && n > 0) {
    // copy workgroups read the release times from device memory: wait until no kernel
    // of this plan still does
    DeviceGuard g(p->device);
    if (g.err != hipSuccess) return hip_fail(g.err, "hipSetDevice");
    for (int par = 0; par < 2; ++par)
      if (p->kernel_pending[par]) CSG_HIP(hipEventSynchronize(p->ev_kernel_done[par]));
    std::vector<uint64_t> ticks(n);
    double t = 0.0;
    for (int32_t i = 0; i < n; ++i) {
      t += delay_us_host[i];
      ticks[i] = static_cast<uint64_t>(t * 100.0);  // 100 MHz wall clock
    }
    CSG_HIP(hipMemcpy(p->d_release_ticks, ticks.data(), ticks.size() * 8, hipMemcpyHostToDevice));
    p->release_set = true;
  }
  return CSG_OK;
}

csg_status csg_ag_gemm(csg_plan* p, void* a_landing, const void* a_staging, const void* b_nk, void* c, csg_mode mode,
                       void* compute_stream, void* copy_stream) {
  if (!p) return fail(CSG_ERR_INVALID, "plan is NULL");
  if (p->op != CSG_AG_GEMM || p->attention()) return fail(CSG_ERR_INVALID, "plan is not an all-gather GEMM plan");
  return consumer_call(p, a_landing, a_staging, b_nk, c, mode, compute_stream, copy_stream);
}

csg_status csg_ag_gemm_noalloc(const csg_schedule* sched, int64_t M, int64_t N, int64_t K, csg_dtype in_dtype,
                               csg_dtype out_dtype, void* a_landing, const void* a_staging, const void* b_nk, void* c,
                               csg_mode mode, int32_t copy_workgroups, int device, void* stream_v) {
  // ---- validation: nothing is queued or allocated before every check has passed
  if (!sched) return fail(CSG_ERR_INVALID, "schedule is NULL");
  const csg::Schedule& s = sched->s;
  if ((in_dtype != CSG_BF16 && in_dtype != CSG_F32) || (out_dtype != CSG_BF16 && out_dtype != CSG_F32))
    return fail(CSG_ERR_INVALID, "unknown dtype");
  if (mode != CSG_MODE_OVERLAP && mode != CSG_MODE_COMPUTE_ONLY && mode != CSG_MODE_COPY_ONLY)
    return fail(CSG_ERR_INVALID, "unknown mode %d", static_cast<int>(mode));
  if (M < 1 || N < 1 || K < 1 || M > 0x7fffffff || N > 0x7fffffff || K > (1 << 22))
    return fail(CSG_ERR_INVALID, "shape out of range");
  if (s.total_rows != M) return fail(CSG_ERR_INVALID, "the schedule's chunks do not cover exactly M rows");
  if (device < 0 || device >= 64) return fail(CSG_ERR_INVALID, "device %d out of range", device);
  if (copy_workgroups == 0) copy_workgroups = kDefaultCopyWorkgroups;
  if (copy_workgroups < 1 || copy_workgroups > 4096) return fail(CSG_ERR_INVALID, "copy_workgroups out of range");
  const bool bf16 = in_dtype == CSG_BF16;
  const int32_t bm = bf16 ? 256 : 64, bn = bf16 ? 256 : 64, bk = bf16 ? 64 : 16;
  const int64_t ib = bf16 ? 2 : 4, ob = out_dtype == CSG_BF16 ? 2 : 4;
  if (K % bk != 0 || N % 4 != 0)
    return fail(CSG_ERR_UNSUPPORTED, "K must be a multiple of %d and N a multiple of 4", bk);
  if (static_cast<int64_t>(std::max(bm, bn)) * K * ib >= (int64_t{1} << 31) ||
      static_cast<int64_t>(bm) * N * ob >= (int64_t{1} << 30))
    return fail(CSG_ERR_UNSUPPORTED, "a tile of A/B or of C exceeds the 32-bit offset range");
  const int32_t n_chunks = static_cast<int32_t>(s.chunks.size());
  if (n_chunks > kNaMaxChunks) return fail(CSG_ERR_UNSUPPORTED, "at most %d chunks", kNaMaxChunks);
  std::vector<int32_t> remote;
  for (int32_t cid : s.order)
    if (!s.chunks[cid].is_local) remote.push_back(cid);
  const bool copies = mode != CSG_MODE_COMPUTE_ONLY && !remote.empty();
  if (!a_landing || !b_nk || !c || (copies && !a_staging)) return fail(CSG_ERR_INVALID, "NULL buffer");
  if (!aligned16(a_landing) || !aligned16(a_staging) || !aligned16(b_nk) || !aligned16(c))
    return fail(CSG_ERR_INVALID, "buffers must be 16-byte aligned");
  const NaLayout L = na_layout();
  if (L.end > csg::kNoAllocScratchBytes) return fail(CSG_ERR_STATE, "scratch layout exceeds the scratch array");
  const csg::KernelKey key{bf16 ? csg::InType::BF16 : csg::InType::F32, out_dtype == CSG_BF16, false, bm, bn, bk,
                           false};
  const int kslot = (bf16 ? 0 : 2) + (out_dtype == CSG_BF16 ? 0 : 1);
  const uint64_t sig = na_signature(s, M, N, K, in_dtype, out_dtype);

  std::lock_guard<std::mutex> lock(g_na_mu);
  NaDevice& nd = g_na[device];
  // ---- the tables of this schedule and shape, on the host (only when they differ from
  //      what the device's scratch holds)
  std::vector<unsigned char> image;
  int32_t n_units = 0, n_items = 0, n_tiles_n = 0;
  bool lines_aligned = true;
  if (nd.sig != sig) {
    csg::TileMap map;
    std::string err = csg::build_tile_map(s, M, N, bm, bn, false, {}, &map);
    if (!err.empty()) return fail(CSG_ERR_INVALID, "%s", err.c_str());
    csg::ExecOptions eo;
    eo.consumer = true;
    eo.K = K;
    eo.in_bytes = ib;
    eo.bk = bk;
    csg::ExecTables et;
    csg::build_exec_tables(s, map, eo, &et);
    std::vector<csg::CopyItem> items;
    std::vector<int32_t> parts;
    csg::build_copy_items(s, remote, K * ib, kCopySlab, &items, &parts);
    n_units = static_cast<int32_t>(et.units.size());
    n_items = static_cast<int32_t>(items.size());
    if (n_units > kNaMaxUnits || static_cast<int64_t>(et.list_ids.size()) > kNaMaxNnz || n_items > kNaMaxItems)
      return fail(CSG_ERR_UNSUPPORTED,
                  "%d tiles, %zu tile-chunk pairs and %d copy slabs of 256 KiB exceed the no-alloc scratch "
                  "(at most %d, %d and %d)",
                  n_units, et.list_ids.size(), n_items, kNaMaxUnits, kNaMaxNnz, kNaMaxItems);
    n_tiles_n = map.n_tiles_n;
    lines_aligned = et.lines_aligned;
    image.assign(L.end - L.tables, 0);
    auto put = [&](size_t at, const void* src, size_t bytes) {
      if (bytes) std::memcpy(image.data() + (at - L.tables), src, bytes);
    };
    put(L.tiles, et.units.data(), et.units.size() * sizeof(csg::TileDesc));
    put(L.list_ptr, et.list_ptr.data(), et.list_ptr.size() * 4);
    put(L.list_ids, et.list_ids.data(), et.list_ids.size() * 4);
    put(L.raster, et.raster.data(), et.raster.size() * 4);
    put(L.list_begin, et.list_begin.data(), et.list_begin.size() * 4);
    put(L.need, et.need.data(), et.need.size() * 4);
    put(L.items, items.data(), items.size() * sizeof(csg::CopyItem));
    put(L.copy_chunk, remote.data(), remote.size() * 4);
    put(L.copy_parts, parts.data(), parts.size() * 4);
    // the ready-value pointers need the device's scratch address: filled in below
  }
  // ---- the device
  DeviceGuard g(device);
  if (g.err != hipSuccess) return hip_fail(g.err, "hipSetDevice");
  if (!nd.checked) {
    char arch[64];
    const csg_status st = csg_device_check(device, arch, sizeof arch);
    if (st != CSG_OK) return st;
    nd.checked = true;
  }
  void* base = nullptr;
  CSG_HIP(csg::noalloc_scratch(device, &base));
  unsigned char* ptr = static_cast<unsigned char*>(base);
  if (!nd.grid[kslot]) CSG_HIP(csg::kernel_grid(key, device, &nd.grid[kslot]));
  hipStream_t stream = static_cast<hipStream_t>(stream_v);
  if (nd.sig != sig) {
    // ready values: a local chunk's is the zero word; a remote chunk's, its ready word
    std::vector<const int64_t*> ready(n_chunks, reinterpret_cast<const int64_t*>(ptr + L.zero));
    for (int32_t cid : remote) ready[cid] = reinterpret_cast<const int64_t*>(ptr + L.kready) + cid;
    std::memcpy(image.data() + (L.ready - L.tables), ready.data(), ready.size() * sizeof(int64_t*));
    nd.sig = 0;  // the scratch holds no valid tables until the copy below is queued
    CSG_HIP(hipMemcpyAsync(ptr + L.tables, image.data(), image.size(), hipMemcpyHostToDevice, stream));
    nd.image.swap(image);
    nd.sig = sig;
    nd.n_units = n_units;
    nd.n_remote = static_cast<int32_t>(remote.size());
    nd.n_items = n_items;
    nd.n_tiles_n = n_tiles_n;
    nd.lines_aligned = lines_aligned;
  }
  nd.calls = nd.calls % 0x3ffffff0u + 1;  // the call number the kernel writes into its consumed words
  const uint32_t epoch = nd.calls;
  // ---- per-call words, then the kernel, on the caller's stream
  csg::PrologueArgs pa{};
  pa.counters = reinterpret_cast<uint32_t*>(ptr + L.counters);
  pa.n_chunks = n_chunks;
  pa.epoch = epoch;
  pa.ticket = reinterpret_cast<uint32_t*>(ptr + L.ticket);
  pa.diag = reinterpret_cast<csg::DeviceDiag*>(ptr + L.diag);
  pa.ready_words = reinterpret_cast<int64_t*>(ptr + L.kready);
  pa.ready_value = mode == CSG_MODE_COMPUTE_ONLY ? 0 : 1;
  pa.copy_done = reinterpret_cast<uint32_t*>(ptr + L.copy_done);
  pa.n_remote = nd.n_remote;
  pa.copy_state = reinterpret_cast<csg::CopyState*>(ptr + L.copy_state);
  CSG_HIP(csg::launch_prologue(pa, stream));
  csg::GemmArgs a{};
  a.A = a_landing;
  a.B = b_nk;
  a.C = c;
  a.M = M;
  a.N = N;
  a.K = K;
  a.tiles = reinterpret_cast<const csg::TileDesc*>(ptr + L.tiles);
  a.list_ptr = reinterpret_cast<const int32_t*>(ptr + L.list_ptr);
  a.list_ids = reinterpret_cast<const int32_t*>(ptr + L.list_ids);
  a.raster = reinterpret_cast<const int32_t*>(ptr + L.raster);
  a.ready = reinterpret_cast<const int64_t* const*>(ptr + L.ready);
  a.counters = pa.counters;
  a.need = reinterpret_cast<const int32_t*>(ptr + L.need);
  a.out_flags = reinterpret_cast<uint32_t*>(ptr + L.out_flags);
  a.ticket = pa.ticket;
  a.list_begin = reinterpret_cast<const int32_t*>(ptr + L.list_begin);
  a.diag = pa.diag;
  a.timeout_ticks = 2000ull * 100000ull;  // 2 s of 100 MHz wall clock per wait
  a.epoch = epoch;
  a.n_tiles = mode == CSG_MODE_COPY_ONLY ? 0 : nd.n_units;
  a.n_chunks = n_chunks;
  a.dynamic_ticket = 1;
  a.steal = 1;
  a.n_tiles_n = mode == CSG_MODE_OVERLAP ? nd.n_tiles_n : 0;
  a.acquire_fresh = (!nd.lines_aligned || reinterpret_cast<uintptr_t>(a_landing) % 128 != 0) ? 1 : 0;
  int32_t grid = nd.grid[kslot];
  if (copies && nd.n_items > 0) {
    a.copy_items = reinterpret_cast<const csg::CopyItem*>(ptr + L.items);
    a.n_copy_items = nd.n_items;
    a.copy_wgs = copy_workgroups;
    a.copy_src = static_cast<const unsigned char*>(a_staging);
    a.copy_dst = static_cast<unsigned char*>(a_landing);
    a.copy_chunk = reinterpret_cast<const int32_t*>(ptr + L.copy_chunk);
    a.copy_parts = reinterpret_cast<const int32_t*>(ptr + L.copy_parts);
    a.copy_done = pa.copy_done;
    a.copy_ready = pa.ready_words;
    a.copy_state = pa.copy_state;
  }
  if (mode == CSG_MODE_COPY_ONLY) {
    if (!copies || nd.n_items == 0) return CSG_OK;  // nothing to move
    grid = std::min(copy_workgroups, grid);
  }
  CSG_HIP(csg::launch_chunk_gemm(key, a, grid, stream, nullptr, nullptr));
  return CSG_OK;
}

csg_status csg_grouped_gemm(csg_plan* p, void* x_landing, const void* x_staging, const void* b_enk, void* c,
                            csg_mode mode, void* compute_stream, void* copy_stream) {
  if (!p) return fail(CSG_ERR_INVALID, "plan is NULL");
  if (p->op != CSG_GROUPED_GEMM || p->attention()) return fail(CSG_ERR_INVALID, "plan is not a grouped GEMM plan");
  return consumer_call(p, x_landing, x_staging, b_enk, c, mode, compute_stream, copy_stream);
}

csg_status csg_gemm_rs(csg_plan* p, const void* a, const void* b_nk, void* c, void* c_outgoing, csg_mode mode,
                       void* compute_stream, void* copy_stream) {
  if (!p) return fail(CSG_ERR_INVALID, "plan is NULL");
  if (p->op != CSG_GEMM_RS || p->attention())
    return fail(CSG_ERR_INVALID, "plan is not a GEMM + reduce-scatter plan");
  if (p->device < 0) return fail(CSG_ERR_STATE, "host-only plan (created with device < 0) cannot run");
  if (!a || !b_nk || !c || (mode != CSG_MODE_COMPUTE_ONLY && !c_outgoing && !p->remote_order.empty()))
    return fail(CSG_ERR_INVALID, "NULL buffer");
  if (!aligned16(a) || !aligned16(b_nk) || !aligned16(c) || !aligned16(c_outgoing))
    return fail(CSG_ERR_INVALID, "buffers must be 16-byte aligned");
  hipStream_t compute = static_cast<hipStream_t>(compute_stream), copy = static_cast<hipStream_t>(copy_stream);
  DeviceGuard g(p->device);
  if (g.err != hipSuccess) return hip_fail(g.err, "hipSetDevice");
  if (p->kernel_copies()) return kernel_copy_call(p, a, nullptr, b_nk, c, c_outgoing, mode, compute);
  CallState cs;
  csg_status st = begin_call(p, mode, &cs);
  if (st != CSG_OK) return st;
  if ((st = launch_prologue_call(p, mode, compute)) != CSG_OK) return st;
  if (mode != CSG_MODE_COPY_ONLY && (st = launch_gemm(p, a, b_nk, c, mode, compute)) != CSG_OK) return st;
  if (mode == CSG_MODE_COMPUTE_ONLY || p->remote_order.empty()) return CSG_OK;
  // copy-only reads the C a previous kernel wrote: that kernel must have finished
  if ((st = ready_copies(p, copy, cs, mode == CSG_MODE_COPY_ONLY)) != CSG_OK) return st;
  const int64_t row_bytes = p->N * out_bytes(p);
  const auto budget = std::chrono::milliseconds(p->cfg.timeout_ms) * 4;
  const Clock::time_point t0 = Clock::now();
  const std::vector<hsa_signal_t>& sigs = call_signals(p);
  p->copies_in_flight = true;
  p->copies_set = p->epoch & 1;
  for (size_t i = 0; i < p->remote_order.size(); ++i) {
    const int32_t cid = p->remote_order[i];
    if (mode == CSG_MODE_OVERLAP) {
      const volatile uint32_t* f = p->h_out_flags + cid;
      while (*f < p->epoch) {
        if (Clock::now() - t0 > budget) {
          p->host_diag = csg_diag{1, cid, -1, *f, p->epoch, 0};
          return fail(CSG_ERR_TIMEOUT, "output chunk %d was not completed in time", cid);
        }
      }
    }
    const csg::ChunkDesc& ch = p->sched.chunks[cid];
    const int64_t off = ch.row_begin * row_bytes;
    // this signal's copy two calls back has long completed (the previous kernel waited
    // for it before rewriting the chunk); check before arming it again
    const hsa_signal_t sig = sigs[i];
    if (csg::sdma_wait(sig, 0, p->cfg.timeout_ms * 4) != 0) {
      p->host_diag = csg_diag{1, cid, -1, 1, p->epoch, 0};
      return fail(CSG_ERR_TIMEOUT, "an earlier copy out of chunk %d did not complete", cid);
    }
    hsa_signal_store_relaxed(sig, 1);
    const size_t bytes = static_cast<size_t>((ch.row_end - ch.row_begin) * row_bytes);
    int pieces = 1;
    const hsa_status_t hs =
        p->cfg.copy_split > 1
            ? p->sdma.copy_pieces(static_cast<char*>(c_outgoing) + off, static_cast<const char*>(c) + off, bytes,
                                  p->cfg.copy_split, sig, p->cfg.timeout_ms * 4, &pieces)
            : p->sdma.copy(static_cast<char*>(c_outgoing) + off, static_cast<const char*>(c) + off, bytes,
                           static_cast<int>(i % p->sdma.count()), nullptr, sig);
    if (hs != HSA_STATUS_SUCCESS) {
      hsa_signal_store_relaxed(sig, 0);
      return fail(CSG_ERR_HIP, "SDMA copy: %s", csg::hsa_error(hs).c_str());
    }
  }
  // the copies complete on their own: the next call's kernel waits for each before
  // rewriting the chunk, and csg_plan_check (or destroy) waits for all of them
  return CSG_OK;
}

csg_status csg_attn_plan_create(int32_t n_heads, int32_t n_kv_heads, int32_t head_dim, int64_t q_rows,
                                const csg_schedule* s, const csg_plan_cfg* cfg, int device, csg_plan** out) {
  if (!out) return fail(CSG_ERR_INVALID, "out is NULL");
  *out = nullptr;
  if (!s) return fail(CSG_ERR_INVALID, "schedule is NULL");
  if (n_heads < 1 || n_kv_heads < 1 || n_heads % n_kv_heads != 0 || head_dim < 1 || q_rows < 1 ||
      q_rows > (int64_t{1} << 30))
    return fail(CSG_ERR_INVALID, "bad attention shape");
  if (head_dim != csg::kAttnHeadDim)
    return fail(CSG_ERR_UNSUPPORTED, "the attention kernel is built for head dimension %d", csg::kAttnHeadDim);
  csg_plan_cfg c = cfg ? *cfg : csg_plan_cfg{};
  if (c.timeout_ms == 0) c.timeout_ms = 2000;
  if (c.copy_engines < 0 || c.copy_engines > 32 || c.timeout_ms < 1 || c.num_workgroups < 0)
    return fail(CSG_ERR_INVALID, "bad plan configuration");
  if (c.copy_backend != CSG_COPY_SDMA || c.split_k > 1 || c.tail_split > 1 || c.tail_wave > 1 || c.intra_order != 0 ||
      c.trace || c.copy_split > 1)
    return fail(CSG_ERR_UNSUPPORTED, "attention plans copy with the SDMA engines and split or trace nothing");
  const csg::Schedule& sch = s->s;
  if (sch.chunks.size() > 4096) return fail(CSG_ERR_UNSUPPORTED, "at most 4096 chunks");
  for (const csg::ChunkDesc& ch : sch.chunks)
    if ((ch.row_end - ch.row_begin) % csg::kAttnBlockKV != 0)
      return fail(CSG_ERR_UNSUPPORTED, "every key/value chunk must hold a multiple of %d rows", csg::kAttnBlockKV);
  if (sch.total_rows > (int64_t{1} << 30) / n_kv_heads) return fail(CSG_ERR_INVALID, "sequence too long");
  csg_plan* p = new (std::nothrow) csg_plan;
  if (!p) return fail(CSG_ERR_NOMEM, "out of host memory");
  p->attn = true;
  p->M = q_rows;
  p->N = n_heads;
  p->K = head_dim;
  p->in_dtype = p->out_dtype = CSG_BF16;
  p->sched = sch;
  p->cfg = c;
  p->at_heads = n_heads;
  p->at_kv_heads = n_kv_heads;
  p->at_q_rows = static_cast<int32_t>(q_rows);
  for (int32_t c_id : p->sched.order)
    if (!p->sched.chunks[c_id].is_local) p->remote_order.push_back(c_id);
  if (device >= 0) {
    char arch[64];
    csg_status st = csg_device_check(device, arch, sizeof arch);
    if (st != CSG_OK) {
      delete p;
      return st;
    }
    p->device = device;
    {
      DeviceGuard g(device);
      hipError_t e = g.err != hipSuccess ? g.err : csg::attn_grid(device, &p->grid);
      if (e != hipSuccess) {
        p->device = -1;
        delete p;
        return hip_fail(e, "occupancy query");
      }
    }
    if (c.num_workgroups > 0) p->grid = c.num_workgroups;
    st = setup_attn_device(p);
    if (st != CSG_OK) {
      std::string msg = g_last_error;
      free_plan_device(p);
      delete p;
      g_last_error = msg;
      return st;
    }
  }
  *out = p;
  return CSG_OK;
}

csg_status csg_ring_attn(csg_plan* p, const void* q, void* k_landing, void* v_landing, const void* k_staging,
                         const void* v_staging, void* o, void* lse, csg_mode mode, void* compute_stream,
                         void* copy_stream) {
  if (!p) return fail(CSG_ERR_INVALID, "plan is NULL");
  if (!p->attention()) return fail(CSG_ERR_INVALID, "plan is not a ring-attention plan");
  if (p->device < 0) return fail(CSG_ERR_STATE, "host-only plan (created with device < 0) cannot run");
  const bool copies = mode != CSG_MODE_COMPUTE_ONLY && !p->remote_order.empty();
  if (!q || !k_landing || !v_landing || !o || !lse || (copies && (!k_staging || !v_staging)))
    return fail(CSG_ERR_INVALID, "NULL buffer");
  if (!aligned16(q) || !aligned16(k_landing) || !aligned16(v_landing) || !aligned16(k_staging) ||
      !aligned16(v_staging) || !aligned16(o) || !aligned16(lse))
    return fail(CSG_ERR_INVALID, "buffers must be 16-byte aligned");
  hipStream_t compute = static_cast<hipStream_t>(compute_stream), copy = static_cast<hipStream_t>(copy_stream);
  DeviceGuard g(p->device);
  if (g.err != hipSuccess) return hip_fail(g.err, "hipSetDevice");
  CallState cs;
  const uint32_t prev_reader = p->last_kernel_epoch;  // the kernel that last read the key/value rows
  csg_status st = begin_call(p, mode, &cs);
  if (st != CSG_OK) return st;
  CopyIssuer issuer(p, k_landing, k_staging, cs.wrapped ? 0u : prev_reader);
  issuer.landing2 = v_landing;
  issuer.staging2 = v_staging;
  if (copies) {
    if ((st = ready_copies(p, copy, cs, false)) != CSG_OK) return st;
    if ((st = issuer.run(false)) != CSG_OK) return st;
  }
  if ((st = launch_prologue_call(p, mode, compute)) != CSG_OK) return st;
  if (mode != CSG_MODE_COPY_ONLY && (st = launch_attn(p, q, k_landing, v_landing, o, lse, compute)) != CSG_OK)
    return st;
  if (!copies) return CSG_OK;
  if ((st = issuer.run(true)) != CSG_OK) return st;
  if (mode == CSG_MODE_COPY_ONLY) return CSG_OK;  // as for the GEMMs: the copies complete on their own
  return finish_copies(p, p->remote_order.size());
}

csg_status csg_gemm_ar(csg_plan* p, const void* a, const void* b_nk, void* c, void* c_outgoing,
                       const void* partials_staging, void* partials_landing, const void* reduced_staging,
                       csg_mode mode, void* compute_stream, void* copy_stream) {
  if (!p) return fail(CSG_ERR_INVALID, "plan is NULL");
  if (p->op != CSG_GEMM_AR || p->attention()) return fail(CSG_ERR_INVALID, "plan is not a GEMM + all-reduce plan");
  if (p->device < 0) return fail(CSG_ERR_STATE, "host-only plan (created with device < 0) cannot run");
  const bool copies = mode != CSG_MODE_COMPUTE_ONLY;
  if (!a || !b_nk || !c || !partials_landing ||
      (copies && (!c_outgoing || !partials_staging || (!reduced_staging && !p->remote_order.empty()))))
    return fail(CSG_ERR_INVALID, "NULL buffer");
  if (!aligned16(a) || !aligned16(b_nk) || !aligned16(c) || !aligned16(c_outgoing) || !aligned16(partials_staging) ||
      !aligned16(partials_landing) || !aligned16(reduced_staging))
    return fail(CSG_ERR_INVALID, "buffers must be 16-byte aligned");
  hipStream_t compute = static_cast<hipStream_t>(compute_stream), copy = static_cast<hipStream_t>(copy_stream);
  DeviceGuard g(p->device);
  if (g.err != hipSuccess) return hip_fail(g.err, "hipSetDevice");
  CallState cs;
  csg_status st = begin_call(p, mode, &cs);
  if (st != CSG_OK) return st;
  p->ar_partials = partials_landing;
  if ((st = launch_prologue_call(p, mode, compute)) != CSG_OK) return st;
  if (mode != CSG_MODE_COPY_ONLY && (st = launch_gemm(p, a, b_nk, c, mode, compute)) != CSG_OK) return st;
  if (!copies) return CSG_OK;
  // the partials land where the previous call's kernel read them, and copy-only sends
  // what a finished kernel wrote: wait for the previous kernel
  if ((st = ready_copies(p, copy, cs, true)) != CSG_OK) return st;
  const int set = p->epoch & 1;
  const int64_t row_bytes = p->N * out_bytes(p);
  const int64_t chunk_bytes = p->ar_chunk_rows * row_bytes;
  const int nq = static_cast<int>(p->ar_own_rows / p->ar_chunk_rows);
  int eng = 0;
  // 1. the other ranks' partial sums of the own shard land, own chunk by own chunk
  const std::vector<hsa_signal_t>& part = p->sig_part[set];
  for (int q = 0; q < nq; ++q)
    for (int j = 0; j < p->ar_peers; ++j) {
      const int64_t off = (static_cast<int64_t>(j) * p->ar_own_rows + static_cast<int64_t>(q) * p->ar_chunk_rows) *
                          row_bytes;
      const hsa_status_t hs =
          p->sdma.copy(static_cast<char*>(partials_landing) + off, static_cast<const char*>(partials_staging) + off,
                       static_cast<size_t>(chunk_bytes), eng++, nullptr, part[static_cast<size_t>(j * nq + q)]);
      // a partial not copied keeps its signal armed: the tiles' bounded waits for it
      // expire and csg_plan_check reports it
      if (hs != HSA_STATUS_SUCCESS) return fail(CSG_ERR_HIP, "SDMA copy of a partial: %s", csg::hsa_error(hs).c_str());
    }
  // 2. in emission order: a non-local chunk is sent (reduce-scatter), then its reduced
  //    rows arrive from their owner into the same rows of c (all-gather), on the same
  //    engine, once the send has read them; an own chunk, reduced by its tiles, is sent
  const std::vector<int32_t>& order = p->sched.order;
  const std::vector<hsa_signal_t>& last = p->sig_ready[set];
  const std::vector<hsa_signal_t>& send = p->sig_send[set];
  const auto budget = std::chrono::milliseconds(p->cfg.timeout_ms) * 4;
  const Clock::time_point t0 = Clock::now();
  for (size_t i = 0; i < order.size(); ++i) {
    const int32_t cid = order[i];
    if (mode == CSG_MODE_OVERLAP) {
      const volatile uint32_t* f = p->h_out_flags + cid;
      while (*f < p->epoch) {
        if (Clock::now() - t0 > budget) {
          p->host_diag = csg_diag{1, cid, -1, *f, p->epoch, 0};
          return fail(CSG_ERR_TIMEOUT, "output chunk %d was not completed in time", cid);
        }
      }
    }
    // this set's signals were last used two calls back (the previous kernel waited for
    // them before rewriting the chunk's rows)
    if (csg::sdma_wait(last[i], 0, p->cfg.timeout_ms * 4) != 0 || csg::sdma_wait(send[i], 0, p->cfg.timeout_ms * 4) != 0) {
      p->host_diag = csg_diag{1, cid, -1, 1, p->epoch, 0};
      return fail(CSG_ERR_TIMEOUT, "an earlier copy of chunk %d did not complete", cid);
    }
    const csg::ChunkDesc& ch = p->sched.chunks[cid];
    const int64_t off = ch.row_begin * row_bytes;
    const size_t bytes = static_cast<size_t>((ch.row_end - ch.row_begin) * row_bytes);
    const int e = eng++;
    hsa_signal_store_relaxed(last[i], 1);
    hsa_status_t hs;
    if (ch.is_local) {
      hs = p->sdma.copy(static_cast<char*>(c_outgoing) + off, static_cast<const char*>(c) + off, bytes, e, nullptr,
                        last[i]);
    } else {
      hsa_signal_store_relaxed(send[i], 1);
      hs = p->sdma.copy(static_cast<char*>(c_outgoing) + off, static_cast<const char*>(c) + off, bytes, e, nullptr,
                        send[i]);
      if (hs == HSA_STATUS_SUCCESS)
        hs = p->sdma.copy(static_cast<char*>(c) + off, static_cast<const char*>(reduced_staging) + off, bytes, e,
                          &send[i], last[i]);
      else
        hsa_signal_store_relaxed(send[i], 0);
    }
    if (hs != HSA_STATUS_SUCCESS) {
      hsa_signal_store_relaxed(last[i], 0);
      return fail(CSG_ERR_HIP, "SDMA copy: %s", csg::hsa_error(hs).c_str());
    }
  }
  // the copies complete on their own: the next call's kernel waits for each chunk's
  // last copy before rewriting its rows, and csg_plan_check waits for all of them
  return CSG_OK;
}

csg_status csg_plan_check(csg_plan* p, csg_diag* out) {
  if (!p) return fail(CSG_ERR_INVALID, "plan is NULL");
  csg_diag d = p->host_diag;
  if (p->device >= 0 && p->epoch > 0) {
    DeviceGuard g(p->device);
    if (g.err != hipSuccess) return hip_fail(g.err, "hipSetDevice");
    CSG_HIP(hipEventSynchronize(p->ev_prologue));
    if (p->kernel_pending[p->epoch & 1]) CSG_HIP(hipEventSynchronize(p->ev_kernel_done[p->epoch & 1]));
    csg_status st = drain_copies(p, true);
    if (st != CSG_OK) return st;
    csg::DeviceDiag dd{};
    CSG_HIP(hipMemcpyAsync(&dd, p->diag(p->epoch & 1), sizeof dd, hipMemcpyDeviceToHost, p->aux));
    CSG_HIP(hipStreamSynchronize(p->aux));
    if (dd.timed_out && !d.timed_out) d = csg_diag{1, dd.chunk, dd.tile, dd.observed, dd.epoch, 0};
    if (!d.timed_out && p->kernel_pending[p->epoch & 1] && dd.units_done != p->expected_units) {
      if (out) *out = d;
      return fail(CSG_ERR_STATE, "the kernel ran %u of %u work units (a die without workgroups?)", dd.units_done,
                  p->expected_units);
    }
  }
  if (out) *out = d;
  if (d.timed_out)
    return fail(CSG_ERR_TIMEOUT, "chunk %d (tile %d) never became ready (value %u, call %u)", d.chunk, d.tile,
                d.observed, d.epoch);
  return CSG_OK;
}

csg_status csg_plan_join(csg_plan* p, void* stream) {
  if (!p) return fail(CSG_ERR_INVALID, "plan is NULL");
  if (p->device < 0) return fail(CSG_ERR_STATE, "host-only plan (created with device < 0) has no copies");
  if (p->kernel_copies() || p->epoch == 0) return CSG_OK;  // no copy outside the plan's kernels
  DeviceGuard g(p->device);
  if (g.err != hipSuccess) return hip_fail(g.err, "hipSetDevice");
  const int set = p->epoch & 1;
  if (p->n_join[set] == 0) return CSG_OK;
  const uint64_t ticks = static_cast<uint64_t>(p->cfg.timeout_ms) * 100000ull;  // 100 MHz wall clock
  CSG_HIP(csg::launch_join(p->d_join[set], p->n_join[set], ticks, p->d_join_flag,
                           static_cast<hipStream_t>(stream)));
  return CSG_OK;
}

csg_status csg_measure_mfma_peak(int device, int32_t iters, double* tflops, double* ms, double* ghz) {
  if (!tflops || iters < 1) return fail(CSG_ERR_INVALID, "NULL output or iters < 1");
  char arch[64];
  csg_status st = csg_device_check(device, arch, sizeof arch);
  if (st != CSG_OK) return st;
  DeviceGuard g(device);
  if (g.err != hipSuccess) return hip_fail(g.err, "hipSetDevice");
  int cus = 0;
  CSG_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device));
  float* sink = nullptr;
  uint64_t* clocks = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  hipStream_t s = nullptr;
  hipError_t e = hipMalloc(&sink, static_cast<size_t>(cus) * 256 * sizeof(float));
  if (e == hipSuccess) e = hipMalloc(&clocks, 2 * sizeof(uint64_t));
  if (e == hipSuccess) e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);
  uint64_t c[2] = {0, 0};
  float t_ms = 0.0f;
  if (e == hipSuccess) e = csg::launch_mfma_peak(cus, iters, sink, clocks, s, e0, e1);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e == hipSuccess) e = hipEventElapsedTime(&t_ms, e0, e1);
  if (e == hipSuccess) e = hipMemcpy(c, clocks, sizeof c, hipMemcpyDeviceToHost);
  for (hipEvent_t ev : {e0, e1})
    if (ev) (void)hipEventDestroy(ev);
  if (s) (void)hipStreamDestroy(s);
  if (sink) (void)hipFree(sink);
  if (clocks) (void)hipFree(clocks);
  if (e != hipSuccess) return hip_fail(e, "MFMA microbenchmark");
  *tflops = t_ms > 0.0f ? csg::mfma_peak_flops(cus, iters) / (t_ms * 1e-3) / 1e12 : 0.0;
  if (ms) *ms = t_ms;
  if (ghz) *ghz = c[1] ? static_cast<double>(c[0]) / (static_cast<double>(c[1]) * 10.0) : 0.0;  // cycles / ns
  return CSG_OK;
}

csg_status csg_plan_trace(csg_plan* p, csg_trace_unit* units_host, int32_t n, int32_t* n_out) {
  if (!p || !units_host || !n_out || n < 0) return fail(CSG_ERR_INVALID, "NULL argument or n < 0");
  *n_out = 0;
  if (p->device < 0 || !p->d_trace) return fail(CSG_ERR_STATE, "plan was not created with tracing");
  if (p->n_launches == 0) return fail(CSG_ERR_STATE, "plan never ran a kernel");
  DeviceGuard g(p->device);
  if (g.err != hipSuccess) return hip_fail(g.err, "hipSetDevice");
  CSG_HIP(hipEventSynchronize(p->ev_k1[(p->n_launches - 1) % kTimingRing]));
  const int32_t m = std::min(n, p->n_units);
  constexpr int W = csg::kTraceWords;
  std::vector<uint64_t> words(static_cast<size_t>(m) * W);
  if (m > 0) {
    CSG_HIP(hipMemcpyAsync(words.data(), p->d_trace, words.size() * sizeof(uint64_t), hipMemcpyDeviceToHost, p->aux));
    CSG_HIP(hipStreamSynchronize(p->aux));
  }
  for (int32_t i = 0; i < m; ++i) {
    const csg::TileDesc& u = p->units[i];
    csg_trace_unit& r = units_host[i];
    r.raster = p->unit_raster[i];
    r.slice = u.slice & 0xffff;
    r.n_slices = u.slice >> 16;
    r.xcd = static_cast<int32_t>(words[W * i + 3] >> 32);
    r.workgroup = static_cast<int32_t>(words[W * i + 3] & 0xffffffffu);
    r.reserved = 0;
    r.t_take = words[W * i + 0];
    r.t_start = words[W * i + 1];
    r.t_end = words[W * i + 2];
    r.cycles = words[W * i + 5] - words[W * i + 4];
  }
  *n_out = m;
  return CSG_OK;
}

csg_status csg_plan_kernel_times(csg_plan* p, float* ms_host, int32_t n, int32_t* n_out) {
  if (!p || !ms_host || !n_out || n < 0) return fail(CSG_ERR_INVALID, "NULL argument or n < 0");
  *n_out = 0;
  if (p->device < 0) return fail(CSG_ERR_STATE, "host-only plan has no kernel launches");
  DeviceGuard g(p->device);
  if (g.err != hipSuccess) return hip_fail(g.err, "hipSetDevice");
  const uint64_t avail = std::min<uint64_t>(p->n_launches, kTimingRing);
  const int32_t m = static_cast<int32_t>(std::min<uint64_t>(avail, static_cast<uint64_t>(n)));
  for (int32_t i = 0; i < m; ++i) {
    const int slot = static_cast<int>((p->n_launches - m + i) % kTimingRing);
    CSG_HIP(hipEventSynchronize(p->ev_k1[slot]));
    CSG_HIP(hipEventElapsedTime(&ms_host[i], p->ev_k0[slot], p->ev_k1[slot]));
  }
  *n_out = m;
  return CSG_OK;
}

void csg_plan_destroy(csg_plan* p) {
  if (!p) return;
  free_plan_device(p);
  delete p;
}

}  // extern "C"
