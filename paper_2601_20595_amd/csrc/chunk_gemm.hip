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
//         (no register staging), double-buffered; LDS rows are 128 bytes with an XOR
//         swizzle of their 16-byte vectors that keeps both the DMA writes and the
//         ds_read_b128 fragment reads free of bank conflicts.
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

// Buffer resource over [base, base + bytes). Callers pass workgroup-uniform values;
// readfirstlane keeps the resource in SGPRs, where buffer instructions need it.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  const int64_t cap = 0x7fffffff;
  const uint64_t p = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(p));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(p >> 32));
  const int n = __builtin_amdgcn_readfirstlane(static_cast<int>(bytes < cap ? bytes : cap));
  void* ub = reinterpret_cast<void*>((static_cast<uint64_t>(hi) << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(ub, 0, n, kBufferDword3);
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

// Next execution position for a workgroup on die `xcd` (thread 0 only): the next
// entry of that die's sub-list, else of the following dies' sub-lists; n_tiles when
// every sub-list is exhausted.
__device__ int next_tile(const GemmArgs& a, uint32_t xcd) {
  for (int d = 0; d < kXcdLists; ++d) {
    const int x = static_cast<int>((xcd + d) % kXcdLists);
    const int len = a.list_begin[x + 1] - a.list_begin[x];
    if (len <= 0) continue;
    if (__hip_atomic_load(a.ticket + x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= static_cast<uint32_t>(len))
      continue;
    const uint32_t t = atomicAdd(a.ticket + x, 1u);
    if (t < static_cast<uint32_t>(len)) return a.list_begin[x] + static_cast<int>(t);
  }
  return a.n_tiles;
}

// Geometry of one output tile as seen by the main loops.
// Ab and Bb point at the unit's first K element of the tile's first row, so a main
// loop reads K steps 0 .. nk-1 of its own unit; the byte ranges end at the last valid
// row's end and bound every load.
struct TileGeom {
  const void* Ab;     // A[row_begin][kt_begin * BK]
  const void* Bb;     // B[col0][kt_begin * BK] (of the tile's group)
  int64_t K;          // row pitch of A and B in elements
  int64_t abytes;     // readable bytes from Ab
  int64_t bbytes;     // readable bytes from Bb
  int arows;          // valid A rows (output rows) of the tile
  int brows;          // valid B rows (output columns) of the tile
  int nk;             // K steps of this unit
};

// ---------------------------------------------------------------------------------
// bf16 main loop: LDS DMA, XOR-swizzled 128-byte rows, BK = 64
// ---------------------------------------------------------------------------------
// One 16-byte-per-lane DMA from a buffer resource into LDS at lds_off + 16 * lane,
// reading byte offset vbase + sadd (vbase per lane, sadd uniform). Issued as inline
// asm so the compiler neither inserts a wait for it in front of every LDS read (it
// cannot tell that the reads target the other stage) nor hoists one offset register
// per load out of the tile loop; the whole offset sits in the VGPR operand, which the
// buffer range check covers. M0 is saved and restored around the load.
__device__ __forceinline__ void dma16(const __amdgpu_buffer_rsrc_t& rs, uint32_t lds_off, int vbase, int sadd) {
  uint32_t saved;
  int voff;
  asm volatile(
      "v_add_u32 %1, %3, %4\n\t"
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "buffer_load_dwordx4 %1, %5, 0 offen lds\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved), "=&v"(voff)
      : "s"(lds_off), "s"(sadd), "v"(vbase), "s"(rs)
      : "memory");
}

__device__ __forceinline__ void wait_dma_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

template <int BM_, int BN_>
struct Bf16Loop {
  static constexpr int BM = BM_, BN = BN_, BK = 64;
  static constexpr int WTM = BM / 2, WTN = BN / 2, MI = WTM / 32, NI = WTN / 32;
  static constexpr int ROWB = 128;                           // bytes per LDS row (64 bf16)
  static constexpr int STAGE_A = BM * ROWB, STAGE_B = BN * ROWB;
  static constexpr int STAGE = STAGE_A + STAGE_B;
  static constexpr int LDS_BYTES = 2 * STAGE;
  static constexpr int A_LOADS = BM / 32, B_LOADS = BN / 32;  // wave DMA issues per stage (8 rows each)
  static_assert(BM % 64 == 0 && BN % 64 == 0, "bf16 tiles are multiples of 64");

  // LDS swizzle: logical 16-byte vector v of tile row r sits at physical vector
  // v ^ swz(r), swz(r) = (r & 7) ^ ((r >> 3) & 1). Any 8 consecutive aligned rows,
  // and the even and the odd rows of any 16 consecutive aligned rows, get distinct
  // swizzles, so a ds_read_b128 of one logical vector by 16 lanes on 16 consecutive
  // rows touches 16 distinct 4-bank groups whether LDS is 32 or 64 banks wide.
  __device__ static int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

  // Issue one stage (the BK columns starting at byte kbase of every row): wave w
  // fills rows [w*BM/4, (w+1)*BM/4) of A and likewise of B. Lane l of an 8-row group
  // writes LDS slot l (row l/8, physical vector l%8), so it fetches logical vector
  // (l%8) ^ swz(row) of that row.
  __device__ static void issue(uint32_t lds_base, int buf, int kbase, const __amdgpu_buffer_rsrc_t& rsA,
                               const __amdgpu_buffer_rsrc_t& rsB, int K, int wave, int lane) {
    const int lr = lane >> 3;
    const int wrow_a = wave * (BM / 4), wrow_b = wave * (BN / 4);
    const uint32_t la = __builtin_amdgcn_readfirstlane(lds_base + buf * STAGE + wrow_a * ROWB);
    const uint32_t lb = __builtin_amdgcn_readfirstlane(lds_base + buf * STAGE + STAGE_A + wrow_b * ROWB);
    // row = group base (a multiple of 8) + lr, so swz(row) = lr ^ ((row >> 3) & 1): the
    // lane part of the offset only depends on the parity of the 8-row group
    const int v_even = lr * K * 2 + (((lane & 7) ^ lr) * 16);
    const int v_odd = lr * K * 2 + (((lane & 7) ^ lr ^ 1) * 16);
#pragma unroll
    for (int q = 0; q < A_LOADS; ++q) {
      const int g8 = wrow_a + q * 8;
      dma16(rsA, la + q * 8 * ROWB, ((g8 >> 3) & 1) ? v_odd : v_even, g8 * K * 2 + kbase);
    }
#pragma unroll
    for (int q = 0; q < B_LOADS; ++q) {
      const int g8 = wrow_b + q * 8;
      dma16(rsB, lb + q * 8 * ROWB, ((g8 >> 3) & 1) ? v_odd : v_even, g8 * K * 2 + kbase);
    }
  }

  __device__ static void run(unsigned char* lds, const TileGeom& g, f32x16 (&acc)[MI][NI], int wave, int lane) {
    const int wm = wave >> 1, wn = wave & 1;
    const __amdgpu_buffer_rsrc_t rsA = make_rsrc(g.Ab, g.abytes);
    const __amdgpu_buffer_rsrc_t rsB = make_rsrc(g.Bb, g.bbytes);
    const int K = static_cast<int>(g.K);
    const int nk = g.nk;
    const uint32_t lds_base =
        __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_ptr_t)lds)));
    const int lrow = lane & 31, lhalf = lane >> 5;
    // byte offset of this lane's fragment row inside a stage; every fragment block
    // starts on a multiple of 32 rows, so the row's swizzle is swz(lane % 32)
    const int a_off = (wm * WTM + lrow) * ROWB;
    const int b_off = STAGE_A + (wn * WTN + lrow) * ROWB;
    const int sw = swz(lrow);

    bf16x8 fa[2][MI], fb[2][NI];  // fragments of two consecutive k sub-steps
    auto load_frags = [&](int set, int buf, int ks) {
      const unsigned char* st = lds + buf * STAGE;
      const int vec = ((ks * 2 + lhalf) ^ sw) * 16;
#pragma unroll
      for (int i = 0; i < MI; ++i)
        fa[set][i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(st + a_off + i * 32 * ROWB + vec));
#pragma unroll
      for (int j = 0; j < NI; ++j)
        fb[set][j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(st + b_off + j * 32 * ROWB + vec));
    };

    issue(lds_base, 0, 0, rsA, rsB, K, wave, lane);
    wait_dma_all();
    __syncthreads();
    load_frags(0, 0, 0);
    for (int t = 0; t < nk; ++t) {
      const int buf = t & 1;
      if (t + 1 < nk) issue(lds_base, buf ^ 1, (t + 1) * BK * 2, rsA, rsB, K, wave, lane);
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        const int cur = ks & 1;
        if (ks + 1 < BK / 16) load_frags(cur ^ 1, buf, ks + 1);  // next sub-step's fragments in flight
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
          for (int j = 0; j < NI; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[cur][j], fa[cur][i], acc[i][j], 0, 0, 0);
        if (ks + 1 < BK / 16) {
          // interleave the next sub-step's LDS reads with this sub-step's MFMAs
#pragma unroll
          for (int q = 0; q < MI + NI; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
          }
          __builtin_amdgcn_sched_group_barrier(0x008, MI * NI - (MI + NI), 0);
        }
      }
      wait_dma_all();   // the next stage has landed in LDS
      __syncthreads();  // and every wave is done with this stage
      if (t + 1 < nk) load_frags(0, buf ^ 1, 0);
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
    const __amdgpu_buffer_rsrc_t rsA = make_rsrc(g.Ab, g.abytes);
    const __amdgpu_buffer_rsrc_t rsB = make_rsrc(g.Bb, g.bbytes);
    const int nk = g.nk;
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
    for (int t = 0; t < nk; ++t) {
      const int buf = t & 1;
      if (t + 1 < nk) load(t + 1);
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
      if (t + 1 < nk) store(buf ^ 1);
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
  uint32_t xcd;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID, 0, 4)" : "=s"(xcd));
  xcd %= kXcdLists;

  for (int iter = 0;; ++iter) {
    __syncthreads();  // everyone is done with s_pos / s_state / LDS of the previous tile
    if (tid == 0) {
      const int pos = a.dynamic_ticket ? next_tile(a, xcd)
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
    // uniform across the workgroup; readfirstlane lets everything derived from it live in SGPRs
    const int pos = __builtin_amdgcn_readfirstlane(s_pos);
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
    const int64_t k0 = static_cast<int64_t>(td.kt_begin) * Loop::BK;
    g.nk = td.kt_end - td.kt_begin;
    g.Ab = static_cast<const unsigned char*>(a.A) + (static_cast<int64_t>(td.row_begin) * a.K + k0) * in_bytes;
    g.Bb = static_cast<const unsigned char*>(a.B) +
           (static_cast<int64_t>(td.group) * a.b_group_stride + col0 * a.K + k0) * in_bytes;
    g.abytes = (static_cast<int64_t>(g.arows) * a.K - k0) * in_bytes;
    g.bbytes = (static_cast<int64_t>(g.brows) * a.K - k0) * in_bytes;

    f32x16 acc[MI][NI];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NI; ++j) acc[i][j] = f32x16{};
    Loop::run(lds, g, acc, wave, lane);

    // Output run (i, j, q) of this thread: accumulator elements 4q..4q+3 of block
    // (i, j), i.e. output row (i * 32 + lane % 32) and columns (j * 32 + 8q +
    // 4 * (lane / 32) + 0..3) of the wave's sub-tile.
    const int N32 = static_cast<int>(a.N);
    const int lrow = lane & 31, lhalf = lane >> 5;
    const int64_t cbase = static_cast<int64_t>(td.row_begin) * a.N + col0;
    auto store_run = [&](int i, int j, int q, const f32x4& f) {
      const int lr = wm * Loop::WTM + i * 32 + lrow;
      const int lc = wn * Loop::WTN + j * 32 + 8 * q + 4 * lhalf;
      if (lr >= g.arows || lc >= g.brows) return;  // N is a multiple of 4: a run is all in or all out
      const int off = lr * N32 + lc;
      if constexpr (kOutBf16)  // v_cvt_pk_bf16_f32: round to nearest even (the default rounding mode)
        *reinterpret_cast<bf16x4*>(static_cast<unsigned short*>(a.C) + cbase + off) = __builtin_convertvector(f, bf16x4);
      else
        *reinterpret_cast<f32x4*>(static_cast<float*>(a.C) + cbase + off) = f;
    };

    const int nslices = td.slice >> 16;
    if (nslices > 1) {
      // Split along K: store this slice's partial sums; the slice that finishes its
      // tile last adds all of them in slice order (so the result does not depend on
      // which slice finished when) and writes the output from those sums.
      constexpr int kVecs = MI * NI * 4;                  // 16-byte vectors per thread
      constexpr int kSliceBytes = kVecs * kThreads * 16;  // one slice of one tile
      // slice layout: vector v of thread t at byte (v * kThreads + t) * 16; addressed
      // through a buffer resource so the per-vector offset is a scalar operand
      const __amdgpu_buffer_rsrc_t rsW =
          make_rsrc(a.ws + static_cast<int64_t>(td.slot) * nslices * (kSliceBytes / 4),
                    static_cast<int64_t>(nslices) * kSliceBytes);
      const int toff = tid * 16;
      const int mine = (td.slice & 0xffff) * kSliceBytes;
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NI; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const f32x4 f = {acc[i][j][4 * q + 0], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, f), rsW, toff,
                                                   mine + ((i * NI + j) * 4 + q) * kThreads * 16, 0);
          }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");  // partials leave this die's L2
      __syncthreads();
      if (tid == 0)
        s_state = (__hip_atomic_fetch_add(a.slot_count + td.slot, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT) ==
                   static_cast<uint32_t>(nslices - 1));
      __syncthreads();
      if (!s_state) continue;
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");  // see the other dies' partials
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NI; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int v = ((i * NI + j) * 4 + q) * kThreads * 16;
            f32x4 sum = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rsW, toff, v, 0));
            for (int sl = 1; sl < nslices; ++sl)
              sum += __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rsW, toff, sl * kSliceBytes + v, 0));
            store_run(i, j, q, sum);
            __builtin_amdgcn_sched_barrier(0);  // one run at a time keeps register use flat
          }
    } else {
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NI; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const f32x4 f = {acc[i][j][4 * q + 0], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
            store_run(i, j, q, f);
            __builtin_amdgcn_sched_barrier(0);  // convert-and-store one run at a time
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
                                                            uint32_t* ticket, DeviceDiag* diag, uint32_t* slot_count,
                                                            int32_t n_slots) {
  const int tid = threadIdx.x;
  for (int i = tid; i < n_slots; i += blockDim.x) slot_count[i] = 0u;
  for (int c = tid; c < n_chunks; c += blockDim.x) {
    if (clear_flags || preset_all)
      __hip_atomic_store(flags + c, preset_all ? epoch : 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    if (counters) counters[c] = 0u;
  }
  if (tid < kXcdLists) ticket[tid] = 0u;
  if (tid == 0) {
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
                           uint32_t* counters, uint32_t* ticket, DeviceDiag* diag, uint32_t* slot_count,
                           int32_t n_slots, hipStream_t stream) {
  hipLaunchKernelGGL(chunk_prologue, dim3(1), dim3(kThreads), 0, stream, flags, n_chunks, epoch, preset_all,
                     clear_flags, counters, ticket, diag, slot_count, n_slots);
  return hipGetLastError();
}

}  // namespace csg
