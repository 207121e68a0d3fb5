// Chunk-scheduled ring attention for gfx950 (CDNA4).
//
// Sequence-parallel attention on one rank: the rank's queries attend to every rank's
// keys and values, which arrive chunk by chunk in ring order (Evaluation, the
// Ring-Attn operator; Section 5.2, tile scheduling that follows the chunk schedule).
// A persistent workgroup takes work units (one head, 128 query rows) from a ticket
// and walks the key/value chunks in arrival order: before a chunk it waits for the
// chunk's ready flag (at most once per chunk and workgroup), then runs the
// flash-attention recurrence over the chunk's keys in blocks of 64. After its last
// block of a chunk it counts the chunk, and the unit that completes the count reports
// the chunk consumed, so the next call may overwrite its rows.
//
// Per wave: 32 query rows, head dimension 128, v_mfma_f32_32x32x16_bf16.
//   scores, transposed: S^T = K . Q^T (first operand K rows from LDS, second operand the
//     wave's queries, kept in registers for the whole unit), so each lane holds the
//     scores of one query row: the row maximum is a maximum over the lane's values and
//     one exchange with lane ^ 32 (which holds the row's other keys);
//   values, transposed: O^T += V^T . P^T. P^T is the score registers converted to bf16;
//     the order in which those registers list the keys is matched by reading V^T rows
//     from LDS in the same order (two 8-byte reads per fragment).
// The K tile is row-major in LDS with 272-byte rows, the V tile is transposed through
// registers into 136-byte rows: both paddings keep the fragment reads free of bank
// conflicts. Scores are scaled into base 2 (exp2), and the log-sum-exp is returned in
// natural log.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "attn.hpp"

namespace csg {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));

constexpr int D = kAttnHeadDim;
constexpr int BQ = kAttnBlockQ;
constexpr int BKV = kAttnBlockKV;
constexpr int kThreads = 256;         // 4 waves x 32 query rows
constexpr int KP = D + 8;             // K tile row pitch (elements): 272 bytes
constexpr int VP = BKV + 4;           // V^T tile row pitch (elements): 136 bytes
constexpr int kMaxAttnChunks = 4096;  // per-workgroup ready cache: one bit per chunk
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kRescaleSlack = 8.0f;  // log2 of the largest weight before a rescale

static_assert(BQ == 32 * (kThreads / 64), "one wave per 32 query rows");

__device__ __forceinline__ int64_t load_ready(const int64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}
__device__ __forceinline__ uint32_t load_flag(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Thread 0: waits until chunk c has landed. 1 if seen ready for the first time in this
// workgroup, 0 if already known, -1 if the wait gave up (timeout, or another
// workgroup's abort).
__device__ int wait_chunk(const AttnArgs& a, int c, int unit, uint32_t* ready_bits) {
  const uint32_t bit = 1u << (c & 31);
  if (ready_bits[c >> 5] & bit) return 0;
  const int64_t* rp = a.ready[c];
  const uint64_t t0 = wall_clock64();
  int64_t v = load_ready(rp);
  while (v != 0) {
    if (load_flag(&a.diag->abort)) return -1;
    if (wall_clock64() - t0 > a.timeout_ticks) {
      if (atomicCAS(&a.diag->timed_out, 0u, 1u) == 0u) {
        a.diag->chunk = c;
        a.diag->tile = unit;
        a.diag->observed = static_cast<uint32_t>(v);
        a.diag->epoch = a.epoch;
      }
      __hip_atomic_store(&a.diag->abort, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      return -1;
    }
    __builtin_amdgcn_s_sleep(32);
    v = load_ready(rp);
  }
  ready_bits[c >> 5] |= bit;
  return 1;
}

// One block of 64 keys (and values) of key/value head g, starting at key row kv0, into
// registers: K as 16-byte row pieces (16 consecutive lanes per row, coalesced); V as
// 16-byte pieces of two adjacent keys (key pair tid % 32, head dims 8 (tid / 32) + 64 j),
// so that the transposing LDS stores write both keys of a head dim in one 4-byte store
// and a wave's stores fall on consecutive addresses.
__device__ __forceinline__ void load_kv(const AttnArgs& a, int g, int kv0, int tid, u32x4_t (&kr)[4],
                                        u32x4_t (&vr)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int p = tid + kThreads * i;
    const int krow = p >> 4, kcol = (p & 15) * 8;
    kr[i] = *reinterpret_cast<const u32x4_t*>(a.K + (static_cast<int64_t>(kv0 + krow) * a.Hkv + g) * D + kcol);
  }
  const int key = 2 * (tid & 31);
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int vcol = ((tid >> 5) + 8 * j) * 8;
      vr[2 * j + t] =
          *reinterpret_cast<const u32x4_t*>(a.V + (static_cast<int64_t>(kv0 + key + t) * a.Hkv + g) * D + vcol);
    }
}

__device__ __forceinline__ void store_kv(uint16_t* sK, uint16_t* sVT, int tid, const u32x4_t (&kr)[4],
                                         const u32x4_t (&vr)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int p = tid + kThreads * i;
    *reinterpret_cast<u32x4_t*>(sK + (p >> 4) * KP + (p & 15) * 8) = kr[i];
  }
  const int key = 2 * (tid & 31);
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int vcol = ((tid >> 5) + 8 * j) * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      // head dim vcol + e of keys key and key + 1
      const uint32_t lo = (vr[2 * j][e >> 1] >> ((e & 1) * 16)) & 0xffffu;
      const uint32_t hi = (vr[2 * j + 1][e >> 1] >> ((e & 1) * 16)) & 0xffffu;
      *reinterpret_cast<uint32_t*>(sVT + (vcol + e) * VP + key) = lo | (hi << 16);
    }
  }
}

// The value of lane ^ 32 of a wave (the other half of a query row's keys), by
// v_permlane32_swap: swapping the halves of two copies of x leaves each lane holding x of
// itself and of lane ^ 32, one in each copy, so their combination is symmetric in the
// two lanes without an LDS round trip.
__device__ __forceinline__ float max_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

}  // namespace

__global__ __launch_bounds__(kThreads, 2) void ring_attn(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t sK[BKV * KP];
  __shared__ __attribute__((aligned(16))) uint16_t sVT[D * VP];
  __shared__ uint32_t ready_bits[kMaxAttnChunks / 32];
  __shared__ int s_unit;
  __shared__ int s_state;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, hlf = lane >> 5;
  if (blockIdx.x == 0 && a.next_ticket) {
    // clear the next call's state set (its prologue, folded into this kernel)
    for (int c = tid; c < a.n_chunks; c += kThreads) a.next_counters[c] = 0u;
    if (tid == 0) {
      a.next_ticket[0] = 0u;
      a.next_diag->timed_out = 0u;
      a.next_diag->chunk = -1;
      a.next_diag->tile = -1;
      a.next_diag->observed = 0u;
      a.next_diag->epoch = a.epoch + 1;
      a.next_diag->abort = 0u;
      a.next_diag->units_done = 0u;
    }
  }
  for (int i = tid; i < kMaxAttnChunks / 32; i += kThreads) ready_bits[i] = 0;
  const int n_qb = (a.Sq + BQ - 1) / BQ;
  const int G = a.H / a.Hkv;
  uint32_t units = 0;

  for (;;) {
    __syncthreads();  // everyone is done with s_unit / s_state / LDS of the previous unit
    if (tid == 0) {
      int u = static_cast<int>(atomicAdd(a.ticket, 1u));
      if (load_flag(&a.diag->abort)) u = a.n_units;
      s_unit = u;
    }
    __syncthreads();
    const int u = __builtin_amdgcn_readfirstlane(s_unit);
    if (u >= a.n_units) break;
    ++units;
    // unit -> (key/value head g, query block, head of g's group): units that run at the
    // same time mostly share key/value heads
    const int per_g = n_qb * G;
    const int g = u / per_g, rem = u - g * per_g;
    const int qb = rem / G, h = g * G + (rem - (rem / G) * G);
    const int q_row = qb * BQ + wave * 32 + l32;
    const bool q_ok = q_row < a.Sq;

    bf16x8_t qf[D / 16];  // second operand of S^T: head dims 16 s + 8 hlf .. + 7
    {
      const uint16_t* qrow = a.Q + (static_cast<int64_t>(q_ok ? q_row : 0) * a.H + h) * D + 8 * hlf;
#pragma unroll
      for (int s = 0; s < D / 16; ++s) {
        const u32x4_t raw = q_ok ? *reinterpret_cast<const u32x4_t*>(qrow + 16 * s) : u32x4_t{0u, 0u, 0u, 0u};
        qf[s] = __builtin_bit_cast(bf16x8_t, raw);
      }
    }
    f32x16_t acc[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db) acc[db] = f32x16_t{};
    float m = -__builtin_inff(), l = 0.0f;

    bool aborted = false;
    for (int pos = 0; pos < a.n_chunks; ++pos) {
      const int c = a.arrival[pos];
      __syncthreads();
      if (tid == 0) s_state = wait_chunk(a, c, u, ready_bits);
      __syncthreads();
      if (s_state < 0) {
        aborted = true;
        break;
      }
      const int r0 = a.chunk_rows[2 * c], r1 = a.chunk_rows[2 * c + 1];
      u32x4_t kr[4], vr[4];
      load_kv(a, g, r0, tid, kr, vr);
      for (int kv0 = r0; kv0 < r1; kv0 += BKV) {
        store_kv(sK, sVT, tid, kr, vr);
        __syncthreads();
        if (kv0 + BKV < r1) load_kv(a, g, kv0 + BKV, tid, kr, vr);  // next block, while this one computes

        // S^T for this block: two 32-key tiles, this wave's 32 query rows
        f32x16_t sc[2] = {f32x16_t{}, f32x16_t{}};
#pragma unroll
        for (int s = 0; s < D / 16; ++s)
#pragma unroll
          for (int kb = 0; kb < 2; ++kb) {
            const bf16x8_t kf = *reinterpret_cast<const bf16x8_t*>(sK + (32 * kb + l32) * KP + 16 * s + 8 * hlf);
            sc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[s], sc[kb], 0, 0, 0);
          }

        // online softmax: this lane holds 32 of the row's 64 scores, lane ^ 32 the rest.
        // The weights are exp2(scale_log2 s - m), m a reference that only moves when the
        // row's scaled maximum exceeds it by more than kRescaleSlack (so weights stay
        // below 2^kRescaleSlack): most blocks leave the accumulators unscaled. Both
        // lanes of a row see the same maximum, so they keep the same reference.
        float mx = -__builtin_inff();
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[kb][r]);
        mx = max_halves(mx) * a.scale_log2;  // the scale is positive
        if (mx > m + kRescaleSlack) {
          const float alpha = __builtin_amdgcn_exp2f(m - mx);  // 0 on the first block
          l *= alpha;
#pragma unroll
          for (int db = 0; db < D / 32; ++db) acc[db] *= alpha;
          m = mx;
        }
        float psum = 0.0f;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            sc[kb][r] = __builtin_amdgcn_exp2f(fmaf(sc[kb][r], a.scale_log2, -m));
            psum += sc[kb][r];
          }
        l += psum;

        // P^T as the second operand, 4 steps of 16 keys: step t takes registers
        // 8 (t % 2) .. + 7 of tile t / 2, which hold keys (t / 2) 32 + (t % 2) 16 +
        // {4 hlf + 0..3, 8 + 4 hlf + 0..3}
        bf16x8_t pb[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const f32x8_t v{sc[t >> 1][8 * (t & 1) + 0], sc[t >> 1][8 * (t & 1) + 1], sc[t >> 1][8 * (t & 1) + 2],
                          sc[t >> 1][8 * (t & 1) + 3], sc[t >> 1][8 * (t & 1) + 4], sc[t >> 1][8 * (t & 1) + 5],
                          sc[t >> 1][8 * (t & 1) + 6], sc[t >> 1][8 * (t & 1) + 7]};
          pb[t] = __builtin_convertvector(v, bf16x8_t);
        }
        // O^T += V^T . P^T, V^T rows read in the same key order
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int kvb = 32 * (t >> 1) + 16 * (t & 1) + 4 * hlf;
#pragma unroll
          for (int db = 0; db < D / 32; ++db) {
            const uint16_t* vrow = sVT + (32 * db + l32) * VP + kvb;
            const u32x2_t lo = *reinterpret_cast<const u32x2_t*>(vrow);
            const u32x2_t hi = *reinterpret_cast<const u32x2_t*>(vrow + 8);
            const bf16x8_t vf = __builtin_bit_cast(bf16x8_t, u32x4_t{lo[0], lo[1], hi[0], hi[1]});
            acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb[t], acc[db], 0, 0, 0);
          }
        }
        __syncthreads();  // this block's LDS reads are done before the next block's stores
      }
      // every load of this chunk by this workgroup has landed (each block's loads are
      // waited for before its LDS stores, and all threads passed the barrier above)
      if (tid == 0) {
        const uint32_t done =
            __hip_atomic_fetch_add(a.counters + c, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) + 1u;
        if (done == static_cast<uint32_t>(a.n_units))
          __hip_atomic_store(a.out_flags + c, a.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      }
    }
    if (aborted) break;

    // O = acc / l over the whole row (both lanes' keys); each lane holds 16 head dims of
    // its row per 32-dim tile, in runs of four
    const float l_tot = sum_halves(l);
    const float inv = 1.0f / l_tot;
    if (q_ok) {
      uint16_t* orow = a.O + (static_cast<int64_t>(q_row) * a.H + h) * D;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int b4 = 0; b4 < 4; ++b4) {
          const f32x4_t v{acc[db][4 * b4 + 0] * inv, acc[db][4 * b4 + 1] * inv, acc[db][4 * b4 + 2] * inv,
                          acc[db][4 * b4 + 3] * inv};
          *reinterpret_cast<u32x2_t*>(orow + 32 * db + 8 * b4 + 4 * hlf) =
              __builtin_bit_cast(u32x2_t, __builtin_convertvector(v, bf16x4_t));
        }
      if (hlf == 0) a.LSE[static_cast<int64_t>(h) * a.Sq + q_row] = (m + log2f(l_tot)) * kLn2;
    }
  }
  if (tid == 0) atomicAdd(&a.diag->units_done, units);
}

int32_t attn_threads() { return kThreads; }

hipError_t launch_ring_attn(const AttnArgs& args, int32_t grid, hipStream_t stream, hipEvent_t start,
                            hipEvent_t stop) {
  hipExtLaunchKernelGGL(ring_attn, dim3(grid), dim3(kThreads), 0, stream, start, stop, 0, args);
  return hipGetLastError();
}

hipError_t attn_grid(int device, int32_t* grid) {
  int cus = 0, per_cu = 0;
  hipError_t e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device);
  if (e != hipSuccess) return e;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(&ring_attn), kThreads, 0);
  if (e != hipSuccess) return e;
  *grid = cus * (per_cu < 1 ? 1 : per_cu);
  return hipSuccess;
}

}  // namespace csg
