// Persistent chunk-scheduled GEMM for gfx950 (CDNA4).
//
// C[M x N] = A[M x K] . B[N x K]^T with one persistent workgroup per co-resident
// slot. Workgroups walk a tile list that the host sorted by chunk arrival
// (consumer ops: all-gather + GEMM, all-to-all + grouped GEMM) or emission
// (producer op: GEMM + reduce-scatter), following the tile-scheduler swizzle of
// Section 5.2:
//   consumer: before a tile, wait until every remote chunk its rows read has a
//             ready flag >= epoch (the copy engine raises it after the chunk's
//             copy). A workgroup remembers the chunks it has seen ready, so it
//             waits at most once per chunk (Section 5.2, minimal synchronization);
//   producer: after a tile, count it against every chunk it wrote; the tile that
//             completes a chunk releases the chunk's flag for the copy engine.
//
// Main loops (256 threads = 2 x 2 waves, each wave a (BM/2) x (BN/2) sub-tile of
// 32 x 32 MFMA blocks):
//   bf16: v_mfma_f32_32x32x16_bf16; tiles stream HBM -> LDS with buffer_load ... lds
//         (no register staging), double-buffered; LDS rows are 128 bytes and the
//         16-byte vectors of row r are stored at vector index (v ^ (r & 7)), which
//         keeps both the DMA writes and the ds_read_b128 fragment reads free of bank
//         conflicts.
//   fp32: v_mfma_f32_32x32x2_f32 with register-staged, padded LDS tiles.
// The MFMA takes the B fragment as its first operand, so each lane ends up with
// four runs of four consecutive output columns of one output row, which the
// epilogue writes as 8-byte (bf16) or 16-byte (fp32) stores.
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace csg {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;

// Buffer resource word 3 for raw (unswizzled, unformatted) buffers on gfx9-family targets.
constexpr int kBufferDword3 = 0x00020000;
constexpr int kThreads = 256;
constexpr int kMaxChunks = 4096;  // per-workgroup ready cache: one bit per chunk

__device__ __forceinline__ uint32_t load_flag(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  const int64_t cap = 0x7fffffff;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes < cap ? bytes : cap),
                                           kBufferDword3);
}

// Waits (thread 0 only) until every listed chunk is ready. Returns 1 if a chunk was
// seen ready for the first time in this workgroup, 0 if all were already known,
// -1 if the wait gave up (timeout here, or another workgroup's abort).
__device__ int wait_chunks(const GemmArgs& a, int pos, uint32_t* ready_bits) {
  int fresh = 0;
  for (int p = a.list_ptr[pos]; p < a.list_ptr[pos + 1]; ++p) {
    const int c = a.list_ids[p];
    const uint32_t bit = 1u << (c & 31);
    if (ready_bits[c >> 5] & bit) continue;
    const uint64_t t0 = wall_clock64();
    uint32_t v = load_flag(a.flags + c);
    while (v < a.epoch) {
      if (load_flag(&a.diag->abort)) return -1;
      if (wall_clock64() - t0 > a.timeout_ticks) {
        if (atomicCAS(&a.diag->timed_out, 0u, 1u) == 0u) {
          a.diag->chunk = c;
          a.diag->tile = a.raster[pos];
          a.diag->observed = v;
          a.diag->epoch = a.epoch;
        }
        __hip_atomic_store(&a.diag->abort, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        return -1;
      }
      __builtin_amdgcn_s_sleep(2);
      v = load_flag(a.flags + c);
    }
    ready_bits[c >> 5] |= bit;
    fresh = 1;
  }
  return fresh;
}

// Geometry of one output tile as seen by the main loops.
struct TileGeom {
  const void* Ab;     // first row of the tile in A
  const void* Bb;     // first row (output column) of the tile in B
  int64_t K;
  int arows;          // valid A rows (output rows) of the tile
  int brows;          // valid B rows (output columns) of the tile
};

// ---------------------------------------------------------------------------------
// bf16 main loop: LDS DMA, XOR-swizzled 128-byte rows, BK = 64
// ---------------------------------------------------------------------------------
template <int BM_, int BN_>
struct Bf16Loop {
  static constexpr int BM = BM_, BN = BN_, BK = 64;
  static constexpr int WTM = BM / 2, WTN = BN / 2, MI = WTM / 32, NI = WTN / 32;
  static constexpr int ROWB = 128;                           // bytes per LDS row (64 bf16)
  static constexpr int STAGE_A = BM * ROWB, STAGE_B = BN * ROWB;
  static constexpr int LDS_BYTES = 2 * (STAGE_A + STAGE_B);
  static constexpr int A_LOADS = BM / 32, B_LOADS = BN / 32;  // wave DMA issues per stage (8 rows each)
  static_assert(BM % 64 == 0 && BN % 64 == 0, "bf16 tiles are multiples of 64");

  // Issue one stage: wave w fills rows [w*BM/4, (w+1)*BM/4) of A and likewise of B.
  __device__ static void issue(unsigned char* lds, int buf, int kt, const __amdgpu_buffer_rsrc_t& rsA,
                               const __amdgpu_buffer_rsrc_t& rsB, int64_t K, int wave, int lane) {
    const int lr = lane >> 3;                       // row inside the 8-row group
    const int logical = (lane & 7) ^ lr;            // logical vector stored at physical slot lane & 7
    const int kbyte = kt * BK * 2 + logical * 16;
    unsigned char* la = lds + buf * (STAGE_A + STAGE_B);
    unsigned char* lb = la + STAGE_A;
#pragma unroll
    for (int q = 0; q < A_LOADS; ++q) {
      const int row = wave * (BM / 4) + q * 8;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsA, (lds_ptr_t)(la + row * ROWB),
                                               16, static_cast<int>((row + lr) * K * 2) + kbyte, 0, 0, 0);
    }
#pragma unroll
    for (int q = 0; q < B_LOADS; ++q) {
      const int row = wave * (BN / 4) + q * 8;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsB, (lds_ptr_t)(lb + row * ROWB),
                                               16, static_cast<int>((row + lr) * K * 2) + kbyte, 0, 0, 0);
    }
  }

  __device__ static void run(unsigned char* lds, const TileGeom& g, f32x16 (&acc)[MI][NI], int wave, int lane) {
    const int wm = wave >> 1, wn = wave & 1;
    const __amdgpu_buffer_rsrc_t rsA = make_rsrc(g.Ab, static_cast<int64_t>(g.arows) * g.K * 2);
    const __amdgpu_buffer_rsrc_t rsB = make_rsrc(g.Bb, static_cast<int64_t>(g.brows) * g.K * 2);
    const int KT = static_cast<int>(g.K / BK);
    const int lrow = lane & 31, lhalf = lane >> 5;
    // byte offset of this lane's fragment row inside a stage; the vector index is
    // XORed with (row & 7) == (lane & 7) because every block starts on a multiple of 8
    const int a_off = (wm * WTM + lrow) * ROWB;
    const int b_off = STAGE_A + (wn * WTN + lrow) * ROWB;
    const int sw = lane & 7;

    issue(lds, 0, 0, rsA, rsB, g.K, wave, lane);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    for (int kt = 0; kt < KT; ++kt) {
      const int buf = kt & 1;
      if (kt + 1 < KT) issue(lds, buf ^ 1, kt + 1, rsA, rsB, g.K, wave, lane);
      const unsigned char* st = lds + buf * (STAGE_A + STAGE_B);
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        const int vec = ((ks * 2 + lhalf) ^ sw) * 16;
        bf16x8 af[MI], bfr[NI];
#pragma unroll
        for (int i = 0; i < MI; ++i)
          af[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(st + a_off + i * 32 * ROWB + vec));
#pragma unroll
        for (int j = 0; j < NI; ++j)
          bfr[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(st + b_off + j * 32 * ROWB + vec));
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
          for (int j = 0; j < NI; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0);
      }
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
    }
  }
};

// ---------------------------------------------------------------------------------
// fp32 main loop: register-staged, padded LDS rows, BK = 16
// ---------------------------------------------------------------------------------
template <int BM_, int BN_>
struct F32Loop {
  static constexpr int BM = BM_, BN = BN_, BK = 16;
  static constexpr int WTM = BM / 2, WTN = BN / 2, MI = WTM / 32, NI = WTN / 32;
  static constexpr int LDK = BK + 4;                      // floats per LDS row
  static constexpr int STAGE_A = BM * LDK * 4, STAGE_B = BN * LDK * 4;
  static constexpr int LDS_BYTES = 2 * (STAGE_A + STAGE_B);
  static constexpr int RPP = kThreads / (BK / 4);         // rows per load pass
  static constexpr int A_PASSES = BM / RPP, B_PASSES = BN / RPP;
  static_assert(BM % RPP == 0 && BN % RPP == 0, "fp32 tile rows");

  __device__ static void run(unsigned char* lds, const TileGeom& g, f32x16 (&acc)[MI][NI], int wave, int lane) {
    const int tid = wave * 64 + lane;
    const int wm = wave >> 1, wn = wave & 1;
    const __amdgpu_buffer_rsrc_t rsA = make_rsrc(g.Ab, static_cast<int64_t>(g.arows) * g.K * 4);
    const __amdgpu_buffer_rsrc_t rsB = make_rsrc(g.Bb, static_cast<int64_t>(g.brows) * g.K * 4);
    const int KT = static_cast<int>(g.K / BK);
    const int vrow = tid / (BK / 4), vcol = (tid % (BK / 4)) * 4;
    const int voff = (vrow * static_cast<int>(g.K) + vcol) * 4;
    const int pass_bytes = RPP * static_cast<int>(g.K) * 4;
    u32x4 ra[A_PASSES], rb[B_PASSES];
    auto load = [&](int kt) {
#pragma unroll
      for (int p = 0; p < A_PASSES; ++p)
        ra[p] = __builtin_amdgcn_raw_buffer_load_b128(rsA, voff + kt * BK * 4 + p * pass_bytes, 0, 0);
#pragma unroll
      for (int p = 0; p < B_PASSES; ++p)
        rb[p] = __builtin_amdgcn_raw_buffer_load_b128(rsB, voff + kt * BK * 4 + p * pass_bytes, 0, 0);
    };
    auto store = [&](int buf) {
      float* sa = reinterpret_cast<float*>(lds + buf * (STAGE_A + STAGE_B));
      float* sb = reinterpret_cast<float*>(lds + buf * (STAGE_A + STAGE_B) + STAGE_A);
#pragma unroll
      for (int p = 0; p < A_PASSES; ++p) *reinterpret_cast<u32x4*>(sa + (vrow + p * RPP) * LDK + vcol) = ra[p];
#pragma unroll
      for (int p = 0; p < B_PASSES; ++p) *reinterpret_cast<u32x4*>(sb + (vrow + p * RPP) * LDK + vcol) = rb[p];
    };
    const int lrow = lane & 31, lhalf = lane >> 5;
    load(0);
    store(0);
    __syncthreads();
    for (int kt = 0; kt < KT; ++kt) {
      const int buf = kt & 1;
      if (kt + 1 < KT) load(kt + 1);
      const float* sa = reinterpret_cast<const float*>(lds + buf * (STAGE_A + STAGE_B));
      const float* sb = reinterpret_cast<const float*>(lds + buf * (STAGE_A + STAGE_B) + STAGE_A);
#pragma unroll
      for (int ks = 0; ks < BK; ks += 2) {
        float af[MI], bfr[NI];
#pragma unroll
        for (int i = 0; i < MI; ++i) af[i] = sa[(wm * WTM + i * 32 + lrow) * LDK + ks + lhalf];
#pragma unroll
        for (int j = 0; j < NI; ++j) bfr[j] = sb[(wn * WTN + j * 32 + lrow) * LDK + ks + lhalf];
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
          for (int j = 0; j < NI; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(bfr[j], af[i], acc[i][j], 0, 0, 0);
      }
      if (kt + 1 < KT) store(buf ^ 1);
      __syncthreads();
    }
  }
};

// ---------------------------------------------------------------------------------
// The persistent kernel
// ---------------------------------------------------------------------------------
template <class Loop, bool kOutBf16, bool kProducer>
__global__ __launch_bounds__(kThreads, 1) void chunk_gemm(GemmArgs a) {
  constexpr int BN = Loop::BN;
  constexpr int MI = Loop::MI, NI = Loop::NI;
  __shared__ __attribute__((aligned(16))) unsigned char lds[Loop::LDS_BYTES];
  __shared__ uint32_t ready_bits[kMaxChunks / 32];
  __shared__ int s_pos;
  __shared__ int s_state;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  for (int i = tid; i < kMaxChunks / 32; i += kThreads) ready_bits[i] = 0;
  const int in_bytes = (Loop::BK == 64) ? 2 : 4;

  for (int iter = 0;; ++iter) {
    __syncthreads();  // everyone is done with s_pos / s_state / LDS of the previous tile
    if (tid == 0) {
      const int pos = a.dynamic_ticket ? static_cast<int>(atomicAdd(a.ticket, 1u))
                                       : static_cast<int>(blockIdx.x) + iter * static_cast<int>(gridDim.x);
      int state = 0;
      if (pos < a.n_tiles) {
        if (load_flag(&a.diag->abort)) state = -1;
        else if (!kProducer) state = wait_chunks(a, pos, ready_bits);
      }
      s_pos = pos;
      s_state = state;
    }
    __syncthreads();
    const int pos = s_pos;
    if (pos >= a.n_tiles || s_state < 0) break;
    // a chunk seen ready for the first time: every wave drops possibly stale cache lines
    if (!kProducer && s_state > 0) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");

    const TileDesc td = a.tiles[pos];
    const int64_t col0 = static_cast<int64_t>(td.n_tile) * BN;
    const int64_t bvalid = a.N - col0;
    TileGeom g;
    g.K = a.K;
    g.arows = td.row_end - td.row_begin;
    g.brows = static_cast<int>(bvalid < BN ? bvalid : BN);
    g.Ab = static_cast<const unsigned char*>(a.A) + static_cast<int64_t>(td.row_begin) * a.K * in_bytes;
    g.Bb = static_cast<const unsigned char*>(a.B) +
           (static_cast<int64_t>(td.group) * a.b_group_stride + col0 * a.K) * in_bytes;

    f32x16 acc[MI][NI];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NI; ++j) acc[i][j] = f32x16{};
    Loop::run(lds, g, acc, wave, lane);

    // epilogue: accumulator element r = 4 * q + t of block (i, j) is output row
    // (i * 32 + lane % 32) and column (j * 32 + 8 * q + 4 * (lane / 32) + t) of the
    // wave's sub-tile
    {
      const int N32 = static_cast<int>(a.N);
      const int lrow = lane & 31, lhalf = lane >> 5;
      const int64_t cbase = static_cast<int64_t>(td.row_begin) * a.N + col0;
#pragma unroll
      for (int i = 0; i < MI; ++i) {
        const int lr = wm * Loop::WTM + i * 32 + lrow;
        if (lr >= g.arows) continue;
#pragma unroll
        for (int j = 0; j < NI; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int lc = wn * Loop::WTN + j * 32 + 8 * q + 4 * lhalf;
            if (lc >= g.brows) continue;  // N is a multiple of 4: a run is all in or all out
            const int off = lr * N32 + lc;
            const f32x16& v = acc[i][j];
            if constexpr (kOutBf16) {
              // v_cvt_pk_bf16_f32: round to nearest even (the default rounding mode)
              const f32x4 f = {v[4 * q + 0], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]};
              *reinterpret_cast<bf16x4*>(static_cast<unsigned short*>(a.C) + cbase + off) =
                  __builtin_convertvector(f, bf16x4);
            } else {
              u32x4 pk;
              pk.x = __float_as_uint(v[4 * q + 0]);
              pk.y = __float_as_uint(v[4 * q + 1]);
              pk.z = __float_as_uint(v[4 * q + 2]);
              pk.w = __float_as_uint(v[4 * q + 3]);
              *reinterpret_cast<u32x4*>(static_cast<float*>(a.C) + cbase + off) = pk;
            }
            __builtin_amdgcn_sched_barrier(0);  // convert-and-store one run at a time
          }
      }
    }

    if constexpr (kProducer) {
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "");  // this wave's C stores reach memory first
      __syncthreads();
      if (tid == 0) {
        for (int p = a.list_ptr[pos]; p < a.list_ptr[pos + 1]; ++p) {
          const int c = a.list_ids[p];
          const uint32_t done =
              __hip_atomic_fetch_add(a.counters + c, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_SYSTEM) + 1u;
          if (done == static_cast<uint32_t>(a.need[c]))
            __hip_atomic_store(a.out_flags + c, a.epoch, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
        }
      }
    }
  }
}

__global__ __launch_bounds__(kThreads) void chunk_prologue(uint32_t* flags, int32_t n_chunks, uint32_t epoch,
                                                            int32_t preset_all, int32_t clear_flags, uint32_t* counters,
                                                            uint32_t* ticket, DeviceDiag* diag) {
  const int tid = threadIdx.x;
  for (int c = tid; c < n_chunks; c += blockDim.x) {
    if (clear_flags || preset_all)
      __hip_atomic_store(flags + c, preset_all ? epoch : 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    if (counters) counters[c] = 0u;
  }
  if (tid == 0) {
    *ticket = 0u;
    diag->timed_out = 0u;
    diag->chunk = -1;
    diag->tile = -1;
    diag->observed = 0u;
    diag->epoch = epoch;
    diag->abort = 0u;
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "");
}

// ---------------------------------------------------------------------------------
// Variant table
// ---------------------------------------------------------------------------------
using LoopBf16_256 = Bf16Loop<256, 256>;
using LoopF32_64 = F32Loop<64, 64>;

template <class Loop, bool kOutBf16, bool kProducer>
static hipError_t launch_one(const GemmArgs& args, int32_t grid, hipStream_t stream) {
  hipLaunchKernelGGL((chunk_gemm<Loop, kOutBf16, kProducer>), dim3(grid), dim3(kThreads), 0, stream, args);
  return hipGetLastError();
}

template <class Loop, bool kOutBf16, bool kProducer>
static const void* kernel_ptr() {
  return reinterpret_cast<const void*>(&chunk_gemm<Loop, kOutBf16, kProducer>);
}

namespace {
struct Variant {
  InType in;
  bool out_bf16;
  bool producer;
  int bm, bn, bk;
  hipError_t (*launch)(const GemmArgs&, int32_t, hipStream_t);
  const void* (*func)();
};

#define CSG_VARIANT(IN, LOOP, OB, PR) \
  Variant { IN, OB, PR, LOOP::BM, LOOP::BN, LOOP::BK, &launch_one<LOOP, OB, PR>, &kernel_ptr<LOOP, OB, PR> }

const Variant kVariants[] = {
    CSG_VARIANT(InType::BF16, LoopBf16_256, true, false),  CSG_VARIANT(InType::BF16, LoopBf16_256, true, true),
    CSG_VARIANT(InType::BF16, LoopBf16_256, false, false), CSG_VARIANT(InType::BF16, LoopBf16_256, false, true),
    CSG_VARIANT(InType::F32, LoopF32_64, false, false),    CSG_VARIANT(InType::F32, LoopF32_64, false, true),
};

const Variant* find_variant(const KernelKey& k) {
  for (const Variant& v : kVariants)
    if (v.in == k.in && v.out_bf16 == k.out_bf16 && v.producer == k.producer && v.bm == k.bm && v.bn == k.bn &&
        v.bk == k.bk)
      return &v;
  return nullptr;
}
}  // namespace

bool kernel_supported(const KernelKey& key) { return find_variant(key) != nullptr; }

int32_t kernel_max_chunks() { return kMaxChunks; }

hipError_t kernel_grid(const KernelKey& key, int device, int32_t* grid) {
  const Variant* v = find_variant(key);
  if (!v) return hipErrorInvalidValue;
  int cus = 0, per_cu = 0;
  hipError_t e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device);
  if (e != hipSuccess) return e;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, v->func(), kThreads, 0);
  if (e != hipSuccess) return e;
  if (per_cu < 1) per_cu = 1;
  *grid = cus * per_cu;
  return hipSuccess;
}

hipError_t launch_chunk_gemm(const KernelKey& key, const GemmArgs& args, int32_t grid, hipStream_t stream) {
  const Variant* v = find_variant(key);
  if (!v) return hipErrorInvalidValue;
  return v->launch(args, grid, stream);
}

hipError_t launch_prologue(uint32_t* flags, int32_t n_chunks, uint32_t epoch, int32_t preset_all, int32_t clear_flags,
                           uint32_t* counters, uint32_t* ticket, DeviceDiag* diag, hipStream_t stream) {
  hipLaunchKernelGGL(chunk_prologue, dim3(1), dim3(kThreads), 0, stream, flags, n_chunks, epoch, preset_all,
                     clear_flags, counters, ticket, diag);
  return hipGetLastError();
}

}  // namespace csg
