// Persistent chunk-scheduled GEMM for gfx950 (CDNA4).
//
// C[M x N] = A[M x K] . B[N x K]^T with one persistent workgroup per co-resident
// slot. Workgroups walk a tile list that the host sorted by chunk arrival
// (consumer ops: all-gather + GEMM, all-to-all + grouped GEMM) or emission
// (producer op: GEMM + reduce-scatter), following the tile-scheduler swizzle of
// Section 5.2:
//   consumer: before a tile, wait until every remote chunk its rows read is ready
//             (its copy's completion signal, which the copy engine brings to 0).
//             A workgroup remembers the chunks it has seen ready, so it waits at
//             most once per chunk (Section 5.2, minimal synchronization);
//   producer: after a tile, count it against every chunk it wrote; the tile that
//             completes a chunk releases the chunk's flag for the copy engine.
//
// Main loops (each wave owns a sub-tile of 32 x 32 output blocks, each one 32 x 32 or
// four 16 x 16 MFMA blocks):
//   bf16: 512 threads = 2 (M) x 4 (N) waves, two per SIMD, so one wave's MFMAs issue
//         while the other waits on LDS or issues its loads; v_mfma_f32_32x32x16_bf16
//         for 256 x 256 and 256 x 224 tiles, v_mfma_f32_16x16x32_bf16 for 128 x 256,
//         256 x 128 and 128 x 128 (the chip holds a higher clock with it, and these
//         tiles have the registers for its twice as many fragments);
//         tiles stream HBM -> LDS with buffer_load ... lds (no register staging)
//         through a ring of K stages: two for 256 x 256 tiles, three for the smaller
//         tiles, whose stages take fewer MFMAs to consume than a load takes to land;
//         LDS rows are 128 bytes with an XOR swizzle of their 16-byte
//         vectors that keeps both the DMA writes and the ds_read_b128 fragment reads
//         free of bank conflicts.
//   fp32: 256 threads = 2 x 2 waves; v_mfma_f32_32x32x2_f32 with register-staged,
//         padded LDS tiles.
// The MFMA takes the B fragment as its first operand, so each lane ends up with runs
// of four consecutive output columns of one output row (the loop's lane_row,
// lane_col, run_row and run_col say where), which the epilogue writes as 8-byte
// (bf16) or 16-byte (fp32) stores.
#include <hip/hip_ext.h>
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
constexpr int kPrologueThreads = 256;
constexpr int kMaxChunks = 4096;  // per-workgroup ready cache: one bit per chunk

__device__ __forceinline__ uint32_t load_flag(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// A chunk's ready value: its copy's completion signal, 0 once the chunk has landed.
__device__ __forceinline__ int64_t load_ready(const int64_t* p) {
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

// Waits (thread 0 only) until every listed chunk is ready: consumers, until its copy
// in has landed; the producer, until the previous call's copy out of its rows has
// completed. Returns 1 if a chunk was seen ready for the first time in this
// workgroup, 0 if all were already known, -1 if the wait gave up (timeout here, or
// another workgroup's abort).
__device__ int wait_chunks(const GemmArgs& a, int pos, uint32_t* ready_bits) {
  int fresh = 0;
  for (int p = a.list_ptr[pos]; p < a.list_ptr[pos + 1]; ++p) {
    const int c = a.list_ids[p];
    const uint32_t bit = 1u << (c & 31);
    if (ready_bits[c >> 5] & bit) continue;
    const uint64_t t0 = wall_clock64();
    const int64_t* rp = a.ready[c];
    int64_t v = load_ready(rp);
    while (v != 0) {
      if (load_flag(&a.diag->abort)) return -1;
      if (wall_clock64() - t0 > a.timeout_ticks) {
        if (atomicCAS(&a.diag->timed_out, 0u, 1u) == 0u) {
          a.diag->chunk = c;
          a.diag->tile = a.raster[pos];
          a.diag->observed = static_cast<uint32_t>(v);
          a.diag->epoch = a.epoch;
        }
        __hip_atomic_store(&a.diag->abort, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        return -1;
      }
      // about 1 us between polls: every waiting workgroup polls words of one page,
      // and faster polling loads that memory channel for no gain
      __builtin_amdgcn_s_sleep(32);
      v = load_ready(rp);
    }
    ready_bits[c >> 5] |= bit;
    fresh = 1;
  }
  return fresh;
}

// GEMM + all-reduce (thread 0 only): waits until the other ranks' partial sums of the
// own-shard tile's rows have landed (each partial chunk's copy brings its value to
// 0). 0 when they have, -1 if the wait gave up.
__device__ int wait_partials(const GemmArgs& a, const TileDesc& td, int pos) {
  const int nq = static_cast<int>(a.own_rows / a.own_chunk_rows);
  const int q0 = static_cast<int>((td.row_begin - a.own_row0) / a.own_chunk_rows);
  const int q1 = static_cast<int>((td.row_end - 1 - a.own_row0) / a.own_chunk_rows);
  for (int j = 0; j < a.n_peers; ++j)
    for (int q = q0; q <= q1; ++q) {
      const int64_t* rp = a.partial_ready[j * nq + q];
      const uint64_t t0 = wall_clock64();
      int64_t v = load_ready(rp);
      while (v != 0) {
        if (load_flag(&a.diag->abort)) return -1;
        if (wall_clock64() - t0 > a.timeout_ticks) {
          if (atomicCAS(&a.diag->timed_out, 0u, 1u) == 0u) {
            a.diag->chunk = a.own_shard * nq + q;
            a.diag->tile = a.raster[pos];
            a.diag->observed = static_cast<uint32_t>(v);
            a.diag->epoch = a.epoch;
          }
          __hip_atomic_store(&a.diag->abort, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
          return -1;
        }
        __builtin_amdgcn_s_sleep(32);
        v = load_ready(rp);
      }
    }
  return 0;
}

// Next execution position for a workgroup on die `xcd` (thread 0 only): the next
// entry of that die's sub-list, else (when stealing is on) of the following dies'
// sub-lists; n_tiles when no list it may take from has entries left.
__device__ int next_tile(const GemmArgs& a, uint32_t xcd) {
  const int dies = a.steal ? kXcdLists : 1;
  for (int d = 0; d < dies; ++d) {
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

// Waits until every vector-memory operation of this wave has completed (loads landed,
// stores acknowledged).
__device__ __forceinline__ void wait_dma_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Waits until at most N of this wave's vector-memory operations are outstanding. Its
// callers (the main loop's ring, the all-reduce's partial-tile ring) issue nothing but
// LDS DMA loads between such waits, and loads complete in issue order, so this lets the
// newest N loads (the stages issued last) stay in flight while every older one has
// landed; an access of the compiler's own in between (a spill) only makes it wait longer. The immediate keeps expcnt and lgkmcnt at
// their maxima (gfx9 encoding: vmcnt bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
template <int N>
__device__ __forceinline__ void wait_dma_keep() {
  static_assert(N >= 0 && N < 64, "vmcnt holds 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Waits until at most `later` groups of PER loads each are outstanding (later is
// workgroup-uniform; more than kMax counts as kMax, less than 1 as none).
template <int PER, int kMax>
__device__ __forceinline__ void wait_dma_stages(int later) {
  if constexpr (kMax >= 1) {
    if (later >= kMax) {
      wait_dma_keep<kMax * PER>();
      return;
    }
    wait_dma_stages<PER, kMax - 1>(later);
  } else {
    wait_dma_all();
  }
}

// Pulls part `part` of `parts` of [0, bytes) of a buffer into the caches: one 4-byte
// load per 128-byte line, written to this wave's 256-byte scratch area of LDS (so no
// register waits for it; the next wait for the wave's loads covers it). Rows that a
// copy engine has just written are not in any cache, and a main loop that finds them
// only in HBM stalls on every K step; the tiles that consume a fresh chunk together
// (one per column tile) each warm one part of its rows first.
template <int kThreads>
__device__ __forceinline__ void warm_lines(const __amdgpu_buffer_rsrc_t& rs, int64_t bytes, int part, int parts,
                                           uint32_t lds_scratch, int tid) {
  const int lines = static_cast<int>(bytes >> 7);
  const int lo = static_cast<int>(static_cast<int64_t>(lines) * part / parts);
  const int hi = static_cast<int>(static_cast<int64_t>(lines) * (part + 1) / parts);
  for (int i = lo + tid; i < hi; i += kThreads) {
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %1\n\t"
        "buffer_load_dword %2, %3, 0 offen lds\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "s"(lds_scratch), "v"(i << 7), "s"(rs)
        : "memory");
  }
}

template <int BM_, int BN_, int WAVES_M_ = 2, int WAVES_N_ = 4, int STAGES_ = 2, int MF_ = 32>
struct Bf16Loop {
  static constexpr int BM = BM_, BN = BN_, BK = 64, IN_BYTES = 2;
  // MFMA shape: 32 = v_mfma_f32_32x32x16_bf16, 16 = v_mfma_f32_16x16x32_bf16 (the same
  // MACs per cycle; under sustained load the chip holds a higher clock with it)
  static constexpr int MF = MF_;
  static_assert(MF == 32 || MF == 16, "MFMA shape");
  // 8 waves, two per SIMD: while one wave of a SIMD waits on LDS or issues its DMA,
  // the other keeps the matrix core busy. Waves are laid out WAVES_M (M) x WAVES_N (N):
  // 2 x 4 by default; 8 x 1 for tiles whose N side (224 = 7 x 32) splits no further.
  static constexpr int WAVES_M = WAVES_M_, WAVES_N = WAVES_N_, WAVES = WAVES_M * WAVES_N, THREADS = WAVES * 64;
  static constexpr int WTM = BM / WAVES_M, WTN = BN / WAVES_N, MI = WTM / 32, NI = WTN / 32;
  static constexpr int ROWB = 128;                           // bytes per LDS row (64 bf16)
  static constexpr int STAGE_A = BM * ROWB, STAGE_B = BN * ROWB;
  static constexpr int STAGE = STAGE_A + STAGE_B;
  // A ring of STAGES stages: STAGES - 1 of them in flight while one is computed on
  static constexpr int STAGES = STAGES_;
  static constexpr int LDS_BYTES = STAGES * STAGE;
  static constexpr int A_GROUPS = BM / 8, B_GROUPS = BN / 8;  // a stage is loaded in groups of 8 rows
  // DMA loads each wave issues per stage, when every wave issues the same number
  static constexpr bool EVEN_ISSUE = A_GROUPS % (2 * WAVES_M_ * WAVES_N_) == 0 && B_GROUPS % (2 * WAVES_M_ * WAVES_N_) == 0;
  static constexpr int DMA_PER_STAGE = (A_GROUPS + B_GROUPS) / (WAVES_M_ * WAVES_N_);
  static_assert(WAVES == 8 && BM % 8 == 0 && BN % 8 == 0 && WTM % 32 == 0 && WTN % 32 == 0, "bf16 tile shape");
  static_assert(STAGES == 2 || ((STAGES == 3 || STAGES == 4) && EVEN_ISSUE && (STAGES - 2) * DMA_PER_STAGE < 64),
                "a deeper ring counts each wave's loads per stage");

  // LDS swizzle: logical 16-byte vector v of tile row r sits at physical vector
  // v ^ swz(r), swz(r) = (r & 7) ^ ((r >> 3) & 1). Any 8 consecutive aligned rows,
  // and the even and the odd rows of any 16 consecutive aligned rows, get distinct
  // swizzles, so a ds_read_b128 of one logical vector by 16 lanes on 16 consecutive
  // rows touches 16 distinct 4-bank groups whether LDS is 32 or 64 banks wide.
  __device__ static int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

  // Output layout. The accumulators of a 32 x 32 block (i, j) of the wave's sub-tile
  // hold four runs q of four consecutive fp32 columns each, at row lane_row(lane) +
  // run_row(i, q) and column lane_col(lane) + run_col(j, q) of the sub-tile. The MFMA
  // takes the B fragment as its first operand, which makes each lane's results runs
  // of columns of one row:
  //   32 x 32 x 16: row lane % 32, columns 4 (lane / 32) + 8 q + 0..3;
  //   16 x 16 x 32: the block is four 16 x 16 blocks, run q = 2 bi + bj; row
  //                 16 bi + lane % 16, columns 16 bj + 4 (lane / 16) + 0..3.
  __device__ static int lane_row(int lane) { return MF == 32 ? (lane & 31) : (lane & 15); }
  __device__ static int lane_col(int lane) { return MF == 32 ? 4 * (lane >> 5) : 4 * (lane >> 4); }
  static constexpr int run_row(int i, int q) { return MF == 32 ? 32 * i : 32 * i + 16 * (q >> 1); }
  static constexpr int run_col(int j, int q) { return MF == 32 ? 32 * j + 8 * q : 32 * j + 16 * (q & 1); }

  // One operand's share of a stage, kGroups groups of 8 rows starting at LDS byte
  // address rows0. When the groups divide evenly, wave w takes a contiguous run of
  // them; otherwise pairs of groups are dealt round robin (pair p to wave p % WAVES).
  // Either way a group's parity, which decides the lane's swizzled offset, is known at
  // compile time.
  template <int kGroups>
  __device__ static void issue_rows(const __amdgpu_buffer_rsrc_t& rs, uint32_t rows0, int wave, int v_even,
                                    int v_odd, int K, int kbase) {
    if constexpr (kGroups % (2 * WAVES) == 0) {
      constexpr int kPer = kGroups / WAVES;  // even
      const int g0 = wave * kPer;
      const uint32_t l0 = __builtin_amdgcn_readfirstlane(rows0 + g0 * 8 * ROWB);
#pragma unroll
      for (int q = 0; q < kPer; ++q) dma16(rs, l0 + q * 8 * ROWB, (q & 1) ? v_odd : v_even, (g0 + q) * 8 * K * 2 + kbase);
    } else {
      static_assert(kGroups % 2 == 0, "an even number of 8-row groups");
      constexpr int kPairs = kGroups / 2;
#pragma unroll
      for (int q = 0; q < (kPairs + WAVES - 1) / WAVES; ++q) {
        const int pr = wave + q * WAVES;
        if (pr < kPairs) {
          const uint32_t l0 = __builtin_amdgcn_readfirstlane(rows0 + pr * 16 * ROWB);
          dma16(rs, l0, v_even, pr * 16 * K * 2 + kbase);
          dma16(rs, l0 + 8 * ROWB, v_odd, (pr * 16 + 8) * K * 2 + kbase);
        }
      }
    }
  }

  // Issue one stage (the BK columns starting at byte kbase of every row), A then B.
  // Lane l of an 8-row group writes LDS slot l (row l/8, physical vector l%8), so it
  // fetches logical vector (l%8) ^ swz(row) of that row; row = 8 g + l/8, so
  // swz(row) = (l/8) ^ (g & 1).
  __device__ static void issue(uint32_t lds_base, int buf, int kbase, const __amdgpu_buffer_rsrc_t& rsA,
                               const __amdgpu_buffer_rsrc_t& rsB, int K, int wave, int lane) {
    const int lr = lane >> 3;
    const uint32_t stage = lds_base + buf * STAGE;
    const int v_even = lr * K * 2 + (((lane & 7) ^ lr) * 16);
    const int v_odd = lr * K * 2 + (((lane & 7) ^ lr ^ 1) * 16);
    issue_rows<A_GROUPS>(rsA, stage, wave, v_even, v_odd, K, kbase);
    issue_rows<B_GROUPS>(rsB, stage + STAGE_A, wave, v_even, v_odd, K, kbase);
  }

  __device__ static void run(unsigned char* lds, const TileGeom& g, f32x16 (&acc)[MI][NI], int wave, int lane) {
    const int wm = wave % WAVES_M, wn = wave / WAVES_M;
    const __amdgpu_buffer_rsrc_t rsA = make_rsrc(g.Ab, g.abytes);
    const __amdgpu_buffer_rsrc_t rsB = make_rsrc(g.Bb, g.bbytes);
    const int K = static_cast<int>(g.K);
    const int nk = g.nk;
    const uint32_t lds_base =
        __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_ptr_t)lds)));
    // A fragment is MF rows of 8 consecutive k values per lane: row lane % MF of the
    // block, 16-byte vector (64 / MF) ks + lane / MF of the row at k sub-step ks (k16
    // sub-steps with 32-row blocks, k32 with 16-row blocks). Every block starts on a
    // multiple of 16 rows and swz repeats every 16 rows, so the row's swizzle is
    // swz(lane % MF).
    constexpr int FI = WTM / MF, FJ = WTN / MF;  // fragments per operand and sub-step
    constexpr int VPS = 64 / MF;                 // 16-byte vectors per k sub-step
    const int lrow = lane % MF, lk = lane / MF;
    const int a_off = (wm * WTM + lrow) * ROWB;
    const int b_off = STAGE_A + (wn * WTN + lrow) * ROWB;
    const int sw = swz(lrow);

    bf16x8 fa[2][FI], fb[2][FJ];  // fragments of two consecutive k sub-steps
    auto load_frags = [&](int set, int buf, int ks) {
      const unsigned char* st = lds + buf * STAGE;
      const int vec = ((ks * VPS + lk) ^ sw) * 16;
#pragma unroll
      for (int i = 0; i < FI; ++i)
        fa[set][i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(st + a_off + i * MF * ROWB + vec));
#pragma unroll
      for (int j = 0; j < FJ; ++j)
        fb[set][j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(st + b_off + j * MF * ROWB + vec));
    };

    issue(lds_base, 0, 0, rsA, rsB, K, wave, lane);
    // Nothing older than the ring's loads stays outstanding (stores of the previous
    // tile included), so the partial waits below count ring loads only.
    wait_dma_all();
#pragma unroll
    for (int s = 1; s < STAGES - 1; ++s)
      if (s < nk) issue(lds_base, s, s * BK * 2, rsA, rsB, K, wave, lane);
    __syncthreads();
    load_frags(0, 0, 0);
    constexpr int kSteps = BK / (512 / MF);  // k sub-steps per stage: 16 (32 x 32) or 32 (16 x 16) each
    constexpr int kMfma = FI * FJ, kReads = FI + FJ;  // per sub-step
    constexpr int kPairs = kMfma < kReads ? kMfma : kReads;
    int buf = 0;  // the ring slot of stage t
    for (int t = 0; t < nk; ++t) {
      const bool more = t + 1 < nk;
      const int next = buf + 1 == STAGES ? 0 : buf + 1;  // slot of stage t + 1
      // Stage t + STAGES - 1 goes into the slot that stage t - 1 used; every wave's
      // reads of it completed before the barrier that ended stage t - 1.
      const bool ahead = t + STAGES - 1 < nk;
      if (ahead) issue(lds_base, buf == 0 ? STAGES - 1 : buf - 1, (t + STAGES - 1) * BK * 2, rsA, rsB, K, wave, lane);
#pragma unroll
      for (int ks = 0; ks < kSteps; ++ks) {
        const int cur = ks & 1;
        if (ks + 1 < kSteps) {
          load_frags(cur ^ 1, buf, ks + 1);  // next sub-step's fragments in flight
        } else {
          // This stage's last fragments are in registers. Wait until the next stage has
          // landed (the stages issued after it may still be in flight) and every wave is
          // done reading this one, then read the next stage's first fragments under this
          // sub-step's MFMAs: the matrix core has queued work on both sides of the
          // barrier instead of draining at it.
          wait_dma_stages<DMA_PER_STAGE, STAGES - 2>(nk - 2 - t);
          __syncthreads();
          if (more) load_frags(cur ^ 1, next, 0);
        }
        if constexpr (MF == 32) {
#pragma unroll
          for (int i = 0; i < MI; ++i)
#pragma unroll
            for (int j = 0; j < NI; ++j)
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[cur][j], fa[cur][i], acc[i][j], 0, 0, 0);
        } else {
          // 16 x 16 block (bi, bj) accumulates into run 2 (bi % 2) + bj % 2 of 32 x 32
          // block (bi / 2, bj / 2)
#pragma unroll
          for (int bi = 0; bi < FI; ++bi)
#pragma unroll
            for (int bj = 0; bj < FJ; ++bj) {
              f32x16& blk = acc[bi >> 1][bj >> 1];
              const int e = 4 * (2 * (bi & 1) + (bj & 1));
              f32x4 c = f32x4{blk[e + 0], blk[e + 1], blk[e + 2], blk[e + 3]};
              c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[cur][bj], fa[cur][bi], c, 0, 0, 0);
              blk[e + 0] = c[0];
              blk[e + 1] = c[1];
              blk[e + 2] = c[2];
              blk[e + 3] = c[3];
            }
        }
        if (ks + 1 < kSteps || more) {
          // interleave the fragment reads in flight with this sub-step's MFMAs
#pragma unroll
          for (int q = 0; q < kPairs; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
          }
          if (kMfma > kPairs) __builtin_amdgcn_sched_group_barrier(0x008, kMfma - kPairs, 0);
          if (kReads > kPairs) __builtin_amdgcn_sched_group_barrier(0x100, kReads - kPairs, 0);
        }
      }
      buf = next;
    }
  }
};

// ---------------------------------------------------------------------------------
// fp32 main loop: register-staged, padded LDS rows, BK = 16
// ---------------------------------------------------------------------------------
template <int BM_, int BN_>
struct F32Loop {
  // output layout: as the bf16 loop's 32 x 32 x 16 one (row lane % 32, runs of four
  // columns at 4 (lane / 32) + 8 q)
  static constexpr int MF = 32;
  __device__ static int lane_row(int lane) { return lane & 31; }
  __device__ static int lane_col(int lane) { return 4 * (lane >> 5); }
  static constexpr int run_row(int i, int) { return 32 * i; }
  static constexpr int run_col(int j, int q) { return 32 * j + 8 * q; }
  static constexpr int BM = BM_, BN = BN_, BK = 16, IN_BYTES = 4;
  static constexpr int WAVES_M = 2, WAVES_N = 2, THREADS = 256;
  static constexpr int WTM = BM / 2, WTN = BN / 2, MI = WTM / 32, NI = WTN / 32;
  static constexpr int LDK = BK + 4;                      // floats per LDS row
  static constexpr int STAGE_A = BM * LDK * 4, STAGE_B = BN * LDK * 4;
  static constexpr int LDS_BYTES = 2 * (STAGE_A + STAGE_B);
  static constexpr int RPP = THREADS / (BK / 4);          // rows per load pass
  static constexpr int A_PASSES = BM / RPP, B_PASSES = BN / RPP;
  static_assert(BM % RPP == 0 && BN % RPP == 0, "fp32 tile rows");

  __device__ static void run(unsigned char* lds, const TileGeom& g, f32x16 (&acc)[MI][NI], int wave, int lane) {
    const int tid = wave * 64 + lane;
    const int wm = wave % WAVES_M, wn = wave / WAVES_M;
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
// Split-K reduction: sum of the S slices' partials of every run, added in slice
// order (((p0 + p1) + p2) + ...), then stored. Runs are handled in batches of B;
// the loads of the next batch are issued before the current batch is added and
// stored, so the reduction pays about one memory latency instead of one per run.
// ---------------------------------------------------------------------------------
constexpr int kDropOffset = 0x7ffffff0;  // buffer offset past every C resource: store dropped
constexpr int kPolicySc0 = 1, kPolicySc1 = 16;  // cache-policy bits of buffer instructions (scope)

// Split-K partial sums. The slices of a tile may run on different dies, whose L2s are
// not coherent with each other: every partial is written through to memory and read
// back past both caches (system-coherent policy, sc0 sc1), so a store that has
// completed is visible to a reader on any die and no cache is written back or
// invalidated.
__device__ __forceinline__ void store_partial(const f32x4& v, const __amdgpu_buffer_rsrc_t& rs, int voff, int soff) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), rs, voff, soff, kPolicySc0 | kPolicySc1);
}
__device__ __forceinline__ f32x4 load_partial(const __amdgpu_buffer_rsrc_t& rs, int voff, int soff) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, voff, soff, kPolicySc0 | kPolicySc1));
}

template <int S, int kRuns, class Load, class Store>
__device__ __forceinline__ void reduce_fixed(Load load, Store store) {
  constexpr int B0 = (8 / S) > 0 ? (8 / S) : 1;
  constexpr int B = (B0 >= 8 && kRuns % 8 == 0) ? 8 : (B0 >= 4 && kRuns % 4 == 0) ? 4 : (B0 >= 2 && kRuns % 2 == 0) ? 2 : 1;
  f32x4 v[2][B][S];
#pragma unroll
  for (int b = 0; b < B; ++b)
#pragma unroll
    for (int s = 0; s < S; ++s) v[0][b][s] = load(s, b);
#pragma unroll
  for (int r0 = 0; r0 < kRuns; r0 += B) {
    const int cur = (r0 / B) & 1;
    if (r0 + B < kRuns) {
#pragma unroll
      for (int b = 0; b < B; ++b)
#pragma unroll
        for (int s = 0; s < S; ++s) v[cur ^ 1][b][s] = load(s, r0 + B + b);
    }
#pragma unroll
    for (int b = 0; b < B; ++b) {
      f32x4 sum = v[cur][b][0];
#pragma unroll
      for (int s = 1; s < S; ++s) sum += v[cur][b][s];
      store(r0 + b, sum);
    }
  }
}

// Two-slice reduction: own (registers) + the other slice's stored partial, run by
// run, with the loads of the next batch of runs in flight while a batch is added.
template <int kRuns, class Load, class Own, class Store>
__device__ __forceinline__ void add_stored_pair(Load load, Own own, Store store) {
  constexpr int B = kRuns % 8 == 0 ? 8 : (kRuns % 4 == 0 ? 4 : 1);
  f32x4 v[2][B];
#pragma unroll
  for (int b = 0; b < B; ++b) v[0][b] = load(b);
#pragma unroll
  for (int r0 = 0; r0 < kRuns; r0 += B) {
    const int cur = (r0 / B) & 1;
    if (r0 + B < kRuns) {
#pragma unroll
      for (int b = 0; b < B; ++b) v[cur ^ 1][b] = load(r0 + B + b);
    }
#pragma unroll
    for (int b = 0; b < B; ++b) store(r0 + b, own(r0 + b) + v[cur][b]);
  }
}

// Waits (thread 0 only) until `others` slices of a split tile have stored their
// partial sums (high half of the tile's slot word). 1 when they have, -1 if the wait
// gave up (timeout, or another workgroup's abort).
__device__ int wait_slices_stored(const GemmArgs& a, const uint32_t* word, int others, int pos) {
  const uint64_t t0 = wall_clock64();
  uint32_t v = __hip_atomic_load(word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  while (static_cast<int>(v >> 16) < others) {
    if (load_flag(&a.diag->abort)) return -1;
    if (wall_clock64() - t0 > a.timeout_ticks) {
      if (atomicCAS(&a.diag->timed_out, 0u, 1u) == 0u) {
        a.diag->chunk = -1;
        a.diag->tile = a.raster[pos];
        a.diag->observed = v >> 16;
        a.diag->epoch = a.epoch;
      }
      __hip_atomic_store(&a.diag->abort, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      return -1;
    }
    __builtin_amdgcn_s_sleep(1);
    v = __hip_atomic_load(word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  return 1;
}

template <int kRuns, class Load, class Store>
__device__ void reduce_slices(int n, Load load, Store store) {
  switch (n) {
    case 2: reduce_fixed<2, kRuns>(load, store); break;
    case 3: reduce_fixed<3, kRuns>(load, store); break;
    case 4: reduce_fixed<4, kRuns>(load, store); break;
    case 5: reduce_fixed<5, kRuns>(load, store); break;
    case 6: reduce_fixed<6, kRuns>(load, store); break;
    case 7: reduce_fixed<7, kRuns>(load, store); break;
    case 8: reduce_fixed<8, kRuns>(load, store); break;
    default:
      for (int r = 0; r < kRuns; ++r) {
        f32x4 sum = load(0, r);
        for (int s = 1; s < n; ++s) sum += load(s, r);
        store(r, sum);
      }
  }
}

// ---------------------------------------------------------------------------------
// Copy workgroups (Section 5.2, realization (4): load/store on specialized
// workgroups, with global-memory signals)
// ---------------------------------------------------------------------------------

// Copy workgroup i (of n) moves items i, i + n, i + 2n, ... (slabs of the chunks in
// arrival order), so the copy workgroups move each chunk together and the chunks
// land in order, with no shared ticket to contend for. A slab moves as 16-byte
// vectors, written through at device scope (sc1: a completed store is visible to
// every die; the readers are this device's tiles). Non-temporal loads and
// system-scope stores measured 30-45 % slower with 16 to 64 copy workgroups. The
// workgroup waits until its stores have completed before it counts the item; the
// one that counts a chunk's last item sets the chunk's ready word to 0. A tile on
// any die that then sees the word at 0 reads the rows from memory: no L2 holds a
// line of them from before (chunks are not read before they are ready, lines left by
// earlier work are dropped at kernel launch, and line-unaligned chunks drop the
// caches on first sight, as with the copy engines). Copy workgroups never wait for
// tiles, so the chunks always land.
template <int kThreads>
__device__ void copy_chunks(const GemmArgs& a, int tid, int copier, int n_copiers) {
  constexpr int U = 8;
  constexpr int kStep = kThreads * 16 * U;
  const uint64_t t0 = a.copy_state->t0;
  int prev = -1;  // the item this workgroup moved last (counted by thread 0 at the next turn)
  // The one thread-0 step of a turn sits right after a barrier and the loop leaves on
  // a uniform value, so every lane of a wave reaches each barrier together.
  for (int item = copier;; item += n_copiers) {
    wait_dma_all();  // this thread's stores of the previous item have completed
    __syncthreads();
    if (tid == 0 && prev >= 0) {
      const CopyItem done_it = a.copy_items[prev];
      const uint32_t done =
          __hip_atomic_fetch_add(a.copy_done + done_it.rpos, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) + 1u;
      if (done == static_cast<uint32_t>(a.copy_parts[done_it.rpos]))
        __hip_atomic_store(a.copy_ready + a.copy_chunk[done_it.rpos], int64_t{0}, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_SYSTEM);
    }
    if (item >= a.n_copy_items) break;
    prev = item;
    const CopyItem it = a.copy_items[item];
    if (a.release_ticks) {
      // the chunk's release time (a simulated peer that is late); bounded by the timeout
      if (tid == 0) {
        const uint64_t due = t0 + a.release_ticks[it.rpos];
        const uint64_t t1 = wall_clock64();
        while (wall_clock64() < due && wall_clock64() - t1 < a.timeout_ticks) __builtin_amdgcn_s_sleep(2);
      }
      __syncthreads();
    }
    const int bytes = __builtin_amdgcn_readfirstlane(it.bytes);
    const int vec_bytes = bytes & ~15;
    const __amdgpu_buffer_rsrc_t rsS = make_rsrc(a.copy_src + it.off, vec_bytes);
    const __amdgpu_buffer_rsrc_t rsD = make_rsrc(a.copy_dst + it.off, vec_bytes);
    // Two register stages: the loads of step k + 1 are in flight while step k is
    // stored. Every 16-byte access is wholly inside the resource or wholly past its
    // end (vec_bytes is a multiple of 16); those past it read 0 and write nothing.
    // The whole offset is the vector operand, which the range check covers.
    auto load_step = [&](u32x4(&v)[U], int base) {
#pragma unroll
      for (int u = 0; u < U; ++u)
        v[u] = __builtin_amdgcn_raw_buffer_load_b128(rsS, base + (u * kThreads + tid) * 16, 0, 0);
    };
    auto store_step = [&](const u32x4(&v)[U], int base) {
#pragma unroll
      for (int u = 0; u < U; ++u)
        __builtin_amdgcn_raw_buffer_store_b128(v[u], rsD, base + (u * kThreads + tid) * 16, 0, kPolicySc1);
    };
    // The next step's loads are issued unconditionally (past the end they read
    // nothing), so the compiler's wait before each store covers only that store's data.
    u32x4 v0[U], v1[U];
    load_step(v0, 0);
    for (int base = 0; base < vec_bytes; base += 2 * kStep) {
      load_step(v1, base + kStep);
      store_step(v0, base);
      load_step(v0, base + 2 * kStep);
      store_step(v1, base + kStep);
    }
    // a tail of 4, 8 or 12 bytes (rows of C whose byte length is not a multiple of 16)
    if (tid < (bytes - vec_bytes) / 4) {
      const uint32_t* src = reinterpret_cast<const uint32_t*>(a.copy_src + it.off + vec_bytes) + tid;
      uint32_t* dst = reinterpret_cast<uint32_t*>(a.copy_dst + it.off + vec_bytes) + tid;
      __hip_atomic_store(dst, *src, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    }
  }
}

// Copies an output tile (rows x row_bytes at pitch bytes, through the resource
// over its rows of C) to dst, the same tile of another buffer with the same pitch:
// 8-byte units (row segments and row starts are multiples of 8 bytes, as N is a
// multiple of 4), reread from L2 where the tile's stores just landed, written
// through to memory. kRowBytes is the widest segment (a full tile row).
template <int kThreads, int kRowBytes>
__device__ void send_tile(const __amdgpu_buffer_rsrc_t& rsC, unsigned char* dst, int rows, int row_bytes, int pitch,
                          int tid) {
  constexpr int kUnitsPerRow = kRowBytes / 8;
  constexpr int U = 8;
  const __amdgpu_buffer_rsrc_t rsD = make_rsrc(dst, static_cast<int64_t>(rows) * pitch);
  const int total = rows * kUnitsPerRow;
  for (int base = 0; base < total; base += kThreads * U) {
    u32x2 v[U];
    int off[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int unit = base + u * kThreads + tid;
      const int row = unit / kUnitsPerRow, col = (unit % kUnitsPerRow) * 8;
      off[u] = (row < rows && col < row_bytes) ? row * pitch + col : kDropOffset;
      v[u] = __builtin_amdgcn_raw_buffer_load_b64(rsC, off[u], 0, kPolicySc0);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) __builtin_amdgcn_raw_buffer_store_b64(v[u], rsD, off[u], 0, kPolicySc0 | kPolicySc1);
  }
}

// ---------------------------------------------------------------------------------
// The persistent kernel
// ---------------------------------------------------------------------------------
template <class Loop, bool kOutBf16, bool kProducer, bool kReduce = false>
__global__ __launch_bounds__(Loop::THREADS, 1) void chunk_gemm(GemmArgs a) {
  constexpr int kThreads = Loop::THREADS;
  constexpr int BN = Loop::BN;
  constexpr int MI = Loop::MI, NI = Loop::NI;
  __shared__ __attribute__((aligned(16))) unsigned char lds[Loop::LDS_BYTES];
  __shared__ uint32_t ready_bits[kMaxChunks / 32];
  __shared__ __attribute__((aligned(16))) uint32_t warm_scratch[kThreads];  // target of warm_lines
  __shared__ int s_pos;
  __shared__ int s_state;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % Loop::WAVES_M, wn = wave / Loop::WAVES_M;
  if (blockIdx.x == 0 && a.next_ticket) {
    // clear the next call's state set (its own prologue, folded into this kernel)
    for (int i = tid; i < a.next_n_slots; i += kThreads) a.next_slot_count[i] = 0u;
    for (int c = tid; c < a.n_chunks; c += kThreads) a.next_counters[c] = 0u;
    if (tid < kXcdLists) a.next_ticket[tid] = 0u;
    if (tid == 0) {
      a.next_diag->timed_out = 0u;
      a.next_diag->chunk = -1;
      a.next_diag->tile = -1;
      a.next_diag->observed = 0u;
      a.next_diag->epoch = a.epoch + 1;
      a.next_diag->abort = 0u;
      a.next_diag->units_done = 0u;
    }
  }
  for (int i = tid; i < kMaxChunks / 32; i += kThreads) ready_bits[i] = 0;
  const int in_bytes = Loop::IN_BYTES;
  uint32_t xcd;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID, 0, 4)" : "=s"(xcd));
  xcd %= kXcdLists;
  uint32_t units = 0;  // work units this workgroup executed (the host checks the total)

  // Workgroups 0 .. copy_wgs - 1 move the chunks, then take tiles too. The dispatcher
  // starts workgroups in index order, so they are running whenever a tile waits.
  const int n_copiers = a.copy_wgs < static_cast<int>(gridDim.x) ? a.copy_wgs : static_cast<int>(gridDim.x);
  if (a.n_copy_items > 0 && static_cast<int>(blockIdx.x) < n_copiers)
    copy_chunks<kThreads>(a, tid, static_cast<int>(blockIdx.x), n_copiers);

  // Static dispatch: workgroup w takes entries slot, slot + G, slot + 2G, ... The
  // dispatcher hands workgroups to the dies round robin (w mod 8), so with
  // slot = (w mod 8) * (G / 8) + w / 8 the workgroups of one die take consecutive
  // entries of every round of G: the tiles of one chunk start together on one die and
  // share its L2 (its A rows, and the B columns of the chunks that follow). Entries
  // from tail_begin on (the K-slices of the last chunks' tiles) go to whichever
  // workgroup asks first: a workgroup whose next static entry lies there takes the next
  // one from a shared ticket instead, so those slices start as soon as their chunk
  // lands rather than behind their fixed workgroup's previous tile.
  const int grid = static_cast<int>(gridDim.x), wg = static_cast<int>(blockIdx.x);
  const int slot = grid % kXcdLists == 0 ? (wg % kXcdLists) * (grid / kXcdLists) + wg / kXcdLists : wg;
  int iter = 0;
  for (;; ++iter) {
    __syncthreads();  // everyone is done with s_pos / s_state / LDS of the previous tile
    if (tid == 0) {
      int pos = a.dynamic_ticket ? next_tile(a, xcd) : slot + iter * grid;
      if (!a.dynamic_ticket && a.tail_begin > 0 && pos >= a.tail_begin) {
        const int t = static_cast<int>(atomicAdd(a.ticket, 1u));
        pos = t < a.n_tiles - a.tail_begin ? a.tail_begin + t : a.n_tiles;
      }
      int state = 0;
      if (pos < a.n_tiles) {
        const uint64_t t_take = a.trace ? wall_clock64() : 0;
        if (load_flag(&a.diag->abort)) state = -1;
        else if (!kProducer) state = wait_chunks(a, pos, ready_bits);
        if (a.trace) {
          a.trace[kTraceWords * pos + 0] = t_take;
          a.trace[kTraceWords * pos + 1] = wall_clock64();
          a.trace[kTraceWords * pos + 3] = (static_cast<uint64_t>(xcd) << 32) | blockIdx.x;
          a.trace[kTraceWords * pos + 4] = clock64();
        }
      }
      s_pos = pos;
      s_state = state;
    }
    __syncthreads();
    // uniform across the workgroup; readfirstlane lets everything derived from it live in SGPRs
    const int pos = __builtin_amdgcn_readfirstlane(s_pos);
    const int state = __builtin_amdgcn_readfirstlane(s_state);
    if (pos >= a.n_tiles || state < 0) break;
    ++units;
    // a chunk seen ready for the first time: every wave drops possibly stale cache
    // lines, unless chunks are line-aligned (then no stale line of a chunk can exist)
    if (!kProducer && state > 0 && a.acquire_fresh) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");

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

    if (!kProducer && state > 0 && a.n_tiles_n > 0) {
      // this workgroup saw one of the tile's chunks land just now: warm its share of
      // the tile's A rows (all K columns), shared with the other column tiles and
      // K-slices
      const int64_t panel = static_cast<int64_t>(g.arows) * a.K * in_bytes;
      const __amdgpu_buffer_rsrc_t rsP =
          make_rsrc(static_cast<const unsigned char*>(a.A) + static_cast<int64_t>(td.row_begin) * a.K * in_bytes, panel);
      const uint32_t scratch = __builtin_amdgcn_readfirstlane(
          static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_ptr_t)warm_scratch)) + wave * 256);
      // the K-slices of a split tile share their tile's part
      const int ns = td.slice >> 16, sl = td.slice & 0xffff;
      warm_lines<kThreads>(rsP, panel, (td.n_tile % a.n_tiles_n) * ns + sl, a.n_tiles_n * ns, scratch, tid);
    }

    f32x16 acc[MI][NI];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NI; ++j) acc[i][j] = f32x16{};
    Loop::run(lds, g, acc, wave, lane);
    if (!kProducer && tid == 0) {
      // every load of this unit has landed (the main loop ends on a wait and a
      // barrier): count the unit against the remote chunks it read, and report a
      // chunk whose last reader this was, so the next call may overwrite its rows
      for (int p = a.list_ptr[pos]; p < a.list_ptr[pos + 1]; ++p) {
        const int c = a.list_ids[p];
        const uint32_t done =
            __hip_atomic_fetch_add(a.counters + c, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) + 1u;
        if (done == static_cast<uint32_t>(a.need[c]))
          __hip_atomic_store(a.out_flags + c, a.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      }
    }

    // Output run r = (i * NI + j) * 4 + q of this thread: accumulator elements
    // 4q..4q+3 of block (i, j), i.e. output row (i * 32 + lane % 32) and columns
    // (j * 32 + 8q + 4 * (lane / 32) + 0..3) of the wave's sub-tile.
    constexpr int kRuns = MI * NI * 4;
    constexpr int kOutBytes = kOutBf16 ? 2 : 4;
    // The producer's C goes straight to memory (system-coherent stores, sc0 sc1): the
    // copy engine reads memory, and a store that completes is then visible to it, so
    // releasing a tile needs no write-back of this die's whole L2. Consumers' C stays
    // in L2 until the kernel's end.
    constexpr int kCStorePolicy = kProducer ? (kPolicySc0 | kPolicySc1) : 0;
    const int N32 = static_cast<int>(a.N);
    // C is written through a buffer resource over the tile's rows; a run outside the
    // valid tile gets a lane offset past the resource's end, and the hardware drops
    // it (the plan keeps BM * N * out_bytes below that offset). No branch, so the
    // epilogue stays one block the compiler can schedule as a whole.
    const __amdgpu_buffer_rsrc_t rsC =
        make_rsrc(static_cast<unsigned char*>(a.C) + (static_cast<int64_t>(td.row_begin) * a.N + col0) * kOutBytes,
                  static_cast<int64_t>(g.arows) * a.N * kOutBytes);
    // the offset of run (i, j, q) is split into a per-lane part (one register), a
    // per-row scalar part (i, q) and a constant that fits the instruction's immediate
    // field (j, q), so no per-run offsets stay live across tiles
    const int vrow = wm * Loop::WTM + Loop::lane_row(lane);  // row of run (i, q): vrow + run_row(i, q)
    const int vcol = wn * Loop::WTN + Loop::lane_col(lane);  // column of run (j, q): vcol + run_col(j, q)
    const int voff_c = (vrow * N32 + vcol) * kOutBytes;
    auto store_run = [&](int r, const f32x4& f) {
      const int i = r / (NI * 4), j = (r / 4) % NI, q = r % 4;
      // N is a multiple of 4: a run is all in or all out
      const bool ok = (vrow + Loop::run_row(i, q) < g.arows) && (vcol + Loop::run_col(j, q) < g.brows);
      const int voff = (ok ? voff_c : kDropOffset) + Loop::run_col(j, q) * kOutBytes;
      const int soff = __builtin_amdgcn_readfirstlane(Loop::run_row(i, q) * N32 * kOutBytes);
      if constexpr (kOutBf16)  // v_cvt_pk_bf16_f32: round to nearest even (the default rounding mode)
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, __builtin_convertvector(f, bf16x4)), rsC, voff,
                                              soff, kCStorePolicy);
      else
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, f), rsC, voff, soff, kCStorePolicy);
    };
    // Producer: the previous call's copy out of a chunk reads the same rows of C this
    // unit is about to write; wait until it has completed (its completion signal reads
    // 0). It normally has, long ago. False if the wait gave up.
    auto wait_previous_copy_out = [&]() -> bool {
      if constexpr (!kProducer) return true;
      __syncthreads();
      if (tid == 0) s_state = wait_chunks(a, pos, ready_bits);
      __syncthreads();
      return __builtin_amdgcn_readfirstlane(s_state) >= 0;
    };
    auto acc_run = [&](int r) -> f32x4 {
      const int i = r / (NI * 4), j = (r / 4) % NI, q = r % 4;
      return f32x4{acc[i][j][4 * q + 0], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
    };

    // A wait of this unit gave up (timeout, or another workgroup's abort): the unit is
    // left unfinished. Every such wait has raised the kernel's abort flag, so each
    // workgroup stops when it takes its next unit; the loop's only exit stays at its top.
    bool skip = false;
    if constexpr (kReduce) {
      // GEMM + all-reduce: a tile of the own shard adds the other ranks' partial sums of
      // its rows (in ascending rank order, in fp32) before its output is stored, so the
      // stored rows are the reduced ones (the reduce-scatter's reduction, fused into the
      // epilogue). Plans with the reduction split no tile and keep tiles inside shards.
      if (td.row_begin >= a.own_row0 && td.row_begin < a.own_row0 + a.own_rows) {
        __syncthreads();
        if (tid == 0) s_state = wait_partials(a, td, pos);
        __syncthreads();
        skip = __builtin_amdgcn_readfirstlane(s_state) < 0;
        const int64_t prow = td.row_begin - a.own_row0;
        if constexpr (kOutBf16 && Loop::BM == 256 && Loop::BN == 256 && kThreads == 512 &&
                      Loop::WAVES_M == 2 && Loop::MI == 4 && Loop::MF == 32) {
          // The peers' partial tiles (256 rows of 512 bytes each) stream through the main
          // loop's LDS in 64-row quarters: quarter k of every peer goes to ring slot k
          // (32 KiB), three quarters in flight while one is added. Each wave stages 8
          // rows of a quarter with row-contiguous 16-byte DMA (two rows per
          // instruction, four instructions); the 16-byte pieces of row r sit at position
          // (piece ^ (r % 32)), so the 32 rows a read instruction touches fall in
          // distinct bank groups. A quarter's rows belong to the four waves of one M
          // half (wm = k / 2), which read their two row blocks of it (i = 2 (k % 2) and
          // 2 (k % 2) + 1) back in the accumulator layout and add them. Peers are added
          // in ascending rank order. Loads past the tile's last row read 0.
          constexpr int kRowB = 512, kQuarterB = 64 * kRowB, kPerUnit = 4;
          const uint32_t lds_base =
              __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_ptr_t)lds)));
          const int pitch = N32 * 2;
          const int units = skip ? 0 : 4 * a.n_peers;
          auto issue_quarter = [&](int j, int k) {
            const __amdgpu_buffer_rsrc_t rsP =
                make_rsrc(a.partials + ((static_cast<int64_t>(j) * a.own_rows + prow) * a.N + col0) * kOutBytes,
                          static_cast<int64_t>(g.arows) * a.N * kOutBytes);
            // The lane's offsets derive from the lane through an empty asm, so they are
            // computed here (a few ALU operations) instead of being hoisted out of the
            // loops and held, or spilled, across them: a spill reload here would make
            // the compiler wait for every load in flight, the ring's included.
            int lw = lane;
            asm volatile("" : "+v"(lw));
            const int qr = lw >> 5, qc = lw & 31;
#pragma unroll
            for (int q2 = 0; q2 < kPerUnit; ++q2) {
              const int lr = wave * 8 + 2 * q2;  // first of this instruction's two rows in the quarter
              const int r = 64 * k + lr + qr;    // tile row of this lane
              const uint32_t l0 = __builtin_amdgcn_readfirstlane(lds_base + k * kQuarterB + lr * kRowB);
              dma16(rsP, l0, r * pitch + ((qc ^ (r & 31)) << 4), 0);
            }
          };
          wait_dma_all();   // only the ring's loads are outstanding from here on
          __syncthreads();  // every wave is done reading the main loop's LDS
          for (int u = 0; u < 3 && u < units; ++u) issue_quarter(u >> 2, u & 3);
          for (int j = 0; j < (units >> 2); ++j) {
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              const int u = 4 * j + k;
              // quarter u has landed; up to two later ones may still be in flight
              wait_dma_stages<kPerUnit, 2>(units - 1 - u);
              __syncthreads();  // every wave's share of quarter u is in, quarter u - 1 is read
              if (u + 3 < units) issue_quarter(j + (k + 3) / 4, (k + 3) & 3);
              if (wm == k / 2) {
#pragma unroll
                for (int r = 0; r < kRuns; ++r) {
                  const int i = r / (NI * 4), jj = (r / 4) % NI, q = r % 4;
                  if (i / 2 != k % 2) continue;
                  const int row = vrow + 32 * i - 64 * k;  // row inside the quarter
                  const int colb = (vcol + 32 * jj + 8 * q) * 2;
                  const u32x2 raw = *reinterpret_cast<const u32x2*>(lds + k * kQuarterB + row * kRowB +
                                                                    (((colb >> 4) ^ (row & 31)) << 4) + (colb & 15));
                  acc[i][jj][4 * q + 0] += __builtin_bit_cast(float, raw.x << 16);
                  acc[i][jj][4 * q + 1] += __builtin_bit_cast(float, raw.x & 0xffff0000u);
                  acc[i][jj][4 * q + 2] += __builtin_bit_cast(float, raw.y << 16);
                  acc[i][jj][4 * q + 3] += __builtin_bit_cast(float, raw.y & 0xffff0000u);
                }
              }
            }
          }
        } else {
        for (int j = 0; j < (skip ? 0 : a.n_peers); ++j) {
          const __amdgpu_buffer_rsrc_t rsP =
              make_rsrc(a.partials + ((static_cast<int64_t>(j) * a.own_rows + prow) * a.N + col0) * kOutBytes,
                        static_cast<int64_t>(g.arows) * a.N * kOutBytes);
#pragma unroll
          for (int r = 0; r < kRuns; ++r) {
            const int i = r / (NI * 4), jj = (r / 4) % NI, q = r % 4;
            const bool ok = (vrow + Loop::run_row(i, q) < g.arows) && (vcol + Loop::run_col(jj, q) < g.brows);
            const int voff = (ok ? voff_c : kDropOffset) + Loop::run_col(jj, q) * kOutBytes;
            const int soff = __builtin_amdgcn_readfirstlane(Loop::run_row(i, q) * N32 * kOutBytes);
            float f[4];
            if constexpr (kOutBf16) {
              const u32x2 raw = __builtin_amdgcn_raw_buffer_load_b64(rsP, voff, soff, 0);
              f[0] = __builtin_bit_cast(float, raw.x << 16);
              f[1] = __builtin_bit_cast(float, raw.x & 0xffff0000u);
              f[2] = __builtin_bit_cast(float, raw.y << 16);
              f[3] = __builtin_bit_cast(float, raw.y & 0xffff0000u);
            } else {
              const f32x4 v = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rsP, voff, soff, 0));
              f[0] = v[0];
              f[1] = v[1];
              f[2] = v[2];
              f[3] = v[3];
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[i][jj][4 * q + e] += f[e];
          }
        }
        }
      }
    }

    const int nslices = td.slice >> 16;
    // false when this unit only left partial sums for another slice of its tile
    bool wrote = true;
    if (skip) {
      wrote = false;
    } else if (nslices == 2) {
      // Split in two along K. The slice that gets here second (low half of the tile's
      // slot word) keeps its partial sums in registers, waits until the other slice has
      // stored its own (high half) and writes the output from the sum of the two
      // (fp32 addition commutes exactly, so the result does not depend on which slice
      // came second); the first slice stores its partials and leaves.
      constexpr int kSliceBytes = kRuns * kThreads * 16;  // one slice of one tile
      const __amdgpu_buffer_rsrc_t rsW = make_rsrc(a.ws + static_cast<int64_t>(td.slot) * (kSliceBytes / 4),
                                                   2 * static_cast<int64_t>(kSliceBytes));
      const int toff = tid * 16;
      const int me = td.slice & 0xffff;
      uint32_t* word = a.slot_count + a.raster[pos];
      if (tid == 0)
        s_state = (__hip_atomic_fetch_add(word, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & 0xffffu) == 1u;
      __syncthreads();
      if (!__builtin_amdgcn_readfirstlane(s_state)) {
#pragma unroll
        for (int r = 0; r < kRuns; ++r) store_partial(acc_run(r), rsW, toff, me * kSliceBytes + r * kThreads * 16);
        wait_dma_all();  // this thread's partials have been written to memory
        __syncthreads();
        if (tid == 0) __hip_atomic_fetch_add(word, 1u << 16, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        wrote = false;
      } else {
        // the other slice has arrived, so it is only storing: a short, bounded wait
        if (tid == 0) s_state = wait_slices_stored(a, word, 1, pos);
        __syncthreads();
        skip = __builtin_amdgcn_readfirstlane(s_state) < 0;
        if (!skip) skip = !wait_previous_copy_out();
        if (!skip) {
          const int other = (1 - me) * kSliceBytes;
          add_stored_pair<kRuns>([&](int r) -> f32x4 { return load_partial(rsW, toff, other + r * kThreads * 16); },
                                 acc_run, store_run);
        }
        wrote = !skip;
      }
    } else if (nslices > 2) {
      // Split along K in more than two: store this slice's partial sums; the slice that
      // finishes its tile last adds all of them in slice order (so the result does not
      // depend on which slice finished when) and writes the output from those sums.
      constexpr int kSliceBytes = kRuns * kThreads * 16;  // one slice of one tile
      // slice layout: run r of thread t at byte (r * kThreads + t) * 16; addressed
      // through a buffer resource so the per-run offset is a scalar operand
      const __amdgpu_buffer_rsrc_t rsW = make_rsrc(a.ws + static_cast<int64_t>(td.slot) * (kSliceBytes / 4),
                                                   static_cast<int64_t>(nslices) * kSliceBytes);
      const int toff = tid * 16;
      const int mine = (td.slice & 0xffff) * kSliceBytes;
#pragma unroll
      for (int r = 0; r < kRuns; ++r) store_partial(acc_run(r), rsW, toff, mine + r * kThreads * 16);
      // waiting for the stores to complete (written through to memory) is the release;
      // the reducer reads memory past its caches
      wait_dma_all();
      __syncthreads();
      if (tid == 0)
        s_state = (__hip_atomic_fetch_add(a.slot_count + a.raster[pos], 1u, __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT) == static_cast<uint32_t>(nslices - 1));
      __syncthreads();
      if (!__builtin_amdgcn_readfirstlane(s_state)) {
        wrote = false;
      } else {
        skip = !wait_previous_copy_out();
        if (!skip) {
          auto load_part = [&](int sl, int r) -> f32x4 { return load_partial(rsW, toff, sl * kSliceBytes + r * kThreads * 16); };
          reduce_slices<kRuns>(nslices, load_part, store_run);
        }
        wrote = !skip;
      }
    } else {
      skip = !wait_previous_copy_out();
      if constexpr (kOutBf16 && Loop::BN == 256 && (Loop::BM == 256 || Loop::BM == 128) && kThreads == 512) {
        // Stored straight from the accumulator layout, one instruction writes 16 bytes
        // of each of 32 rows: partial lines, which for the producer (written through to
        // memory) the memory side takes at twice their size. The tile is staged in LDS
        // instead (rows of 512 bytes, 16-byte piece p of row r at position p ^ (r % 32),
        // the same conflict-free layout as the all-reduce staging) and written out as
        // whole rows, two per instruction.
        if (!skip) {
          constexpr int kRowB = 512;
          static_assert(Loop::BM * kRowB <= Loop::LDS_BYTES, "the staged tile fits the main loop's LDS");
          // the lane index passes through an empty asm, so the addresses derived from it
          // are computed here, per tile, instead of being hoisted out of the tile loop
          // and held in registers across the main loop
          int lw = lane;
          asm volatile("" : "+v"(lw));
          const int l_row = wm * Loop::WTM + Loop::lane_row(lw);  // the lane's row of run (0, q = 0)
          const int l_col2 = (wn * Loop::WTN + Loop::lane_col(lw)) * 2;  // its byte in the row, run (0, 0)
          __syncthreads();  // every wave is done reading LDS
#pragma unroll
          for (int r = 0; r < kRuns; ++r) {
            // run (i, j, q): 8 bytes at row l_row + run_row(i, q), byte l_col2 + 2 run_col(j, q)
            // of the row, that is 16-byte piece (byte / 16) at position piece ^ (row % 32)
            const int i = r / (NI * 4), j = (r / 4) % NI, q = r % 4;
            const int row = l_row + Loop::run_row(i, q);
            const int colb = l_col2 + 2 * Loop::run_col(j, q);
            *reinterpret_cast<u32x2*>(lds + row * kRowB + ((((colb >> 4) ^ row) & 31) << 4) + (colb & 15)) =
                __builtin_bit_cast(u32x2, __builtin_convertvector(acc_run(r), bf16x4));
            __builtin_amdgcn_sched_barrier(0);  // convert-and-write one run at a time
          }
          __syncthreads();
          const int pr = lw >> 5, pc = lw & 31;
          const int c8 = pc * 8;  // first of the piece's 8 columns
          const int vlane = pr * N32 * 2 + pc * 16;
          constexpr int kRowsPerWave = Loop::BM / 8;
#pragma unroll
          for (int q2 = 0; q2 < kRowsPerWave / 2; ++q2) {
            const int row0 = wave * kRowsPerWave + 2 * q2;  // this instruction's rows: row0 + pr
            const u32x4 v =
                *reinterpret_cast<const u32x4*>(lds + (row0 + pr) * kRowB + ((pc ^ ((row0 + pr) & 31)) << 4));
            const int voff = row0 + pr < g.arows ? vlane : kDropOffset;
            const int soff = __builtin_amdgcn_readfirstlane(row0 * N32 * 2);
            if (c8 + 8 <= g.brows)
              __builtin_amdgcn_raw_buffer_store_b128(v, rsC, voff, soff, kCStorePolicy);
            else if (c8 + 4 <= g.brows)  // N is a multiple of 4: a half piece ends the row
              __builtin_amdgcn_raw_buffer_store_b64(u32x2{v.x, v.y}, rsC, voff, soff, kCStorePolicy);
          }
        }
      } else if (!skip) {
#pragma unroll
        for (int r = 0; r < kRuns; ++r) {
          store_run(r, acc_run(r));
          __builtin_amdgcn_sched_barrier(0);  // convert-and-store one run at a time
        }
      }
      wrote = !skip;
    }

    if (kProducer && wrote) {
      // This wave's C stores (system-coherent, written through to memory) have
      // completed before the workgroup counts the tile. The counter and flag updates
      // are relaxed system-scope atomics, performed at the memory side; they are
      // ordered after the stores by the wait and the barrier, and the tile completing
      // a chunk raises its flag only after every other tile of the chunk counted
      // itself, each after its own stores completed. No cache is written back or
      // invalidated.
      wait_dma_all();
      __syncthreads();
      if (a.C2 != nullptr && a.chunk_sent[a.list_ids[a.list_ptr[pos]]] != 0) {
        // Sending from the epilogue (Section 5.2, load/store on the computing
        // workgroup): the tile's output rows, just stored, go to the outgoing buffer
        // too (plans that send this way keep every tile inside one chunk), and count
        // as sent once these stores have completed as well
        send_tile<kThreads, BN * kOutBytes>(rsC, static_cast<unsigned char*>(a.C2) +
                                                     (static_cast<int64_t>(td.row_begin) * a.N + col0) * kOutBytes,
                                            g.arows, g.brows * kOutBytes, N32 * kOutBytes, tid);
        wait_dma_all();
        __syncthreads();
      }
      if (tid == 0) {
        for (int p = a.list_ptr[pos]; p < a.list_ptr[pos + 1]; ++p) {
          const int c = a.list_ids[p];
          const uint32_t done =
              __hip_atomic_fetch_add(a.counters + c, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) + 1u;
          if (done == static_cast<uint32_t>(a.need[c]))
            __hip_atomic_store(a.out_flags + c, a.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        }
      }
    }
    if (a.trace && tid == 0) {
      a.trace[kTraceWords * pos + 2] = wall_clock64();
      a.trace[kTraceWords * pos + 5] = clock64();
    }
  }
  if (tid == 0) atomicAdd(&a.diag->units_done, units);
}

__global__ __launch_bounds__(kPrologueThreads) void chunk_prologue(PrologueArgs p) {
  const int tid = threadIdx.x;
  for (int i = tid; i < p.n_slots; i += blockDim.x) p.slot_count[i] = 0u;
  if (p.counters)
    for (int c = tid; c < p.n_chunks; c += blockDim.x) p.counters[c] = 0u;
  if (p.ready_words)
    for (int c = tid; c < p.n_chunks; c += blockDim.x) p.ready_words[c] = p.ready_value;
  if (p.copy_done)
    for (int i = tid; i < p.n_remote; i += blockDim.x) p.copy_done[i] = 0u;
  if (tid < kXcdLists) p.ticket[tid] = 0u;
  if (tid == 0) {
    p.diag->timed_out = 0u;
    p.diag->chunk = -1;
    p.diag->tile = -1;
    p.diag->observed = 0u;
    p.diag->epoch = p.epoch;
    p.diag->abort = 0u;
    p.diag->units_done = 0u;
    if (p.copy_state) p.copy_state->t0 = wall_clock64();  // release times count from here
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "");
}

// ---------------------------------------------------------------------------------
// Variant table
// ---------------------------------------------------------------------------------
using LoopBf16_256 = Bf16Loop<256, 256>;
// Tiles smaller than 256 x 256 finish a stage's MFMAs sooner than its DMA lands when
// only one stage is in flight; a ring of three keeps two in flight (48 KiB stages: three
// fit the 160 KiB of LDS). Their loops issue 16 x 16 x 32 MFMAs.
using LoopBf16_256x128 = Bf16Loop<256, 128, 2, 4, 3, 16>;
using LoopBf16_128x256 = Bf16Loop<128, 256, 2, 4, 3, 16>;
using LoopBf16_128 = Bf16Loop<128, 128, 2, 4, 3, 16>;
using LoopBf16_256x224 = Bf16Loop<256, 224, 8, 1>;
using LoopF32_64 = F32Loop<64, 64>;

// The timing events (either may be null) take the dispatch's own start and end
// timestamps, not those of separate markers queued around it.
template <class Loop, bool kOutBf16, bool kProducer, bool kReduce>
static hipError_t launch_one(const GemmArgs& args, int32_t grid, hipStream_t stream, hipEvent_t start,
                             hipEvent_t stop) {
  hipExtLaunchKernelGGL((chunk_gemm<Loop, kOutBf16, kProducer, kReduce>), dim3(grid), dim3(Loop::THREADS), 0, stream,
                        start, stop, 0, args);
  return hipGetLastError();
}

template <class Loop, bool kOutBf16, bool kProducer, bool kReduce>
static const void* kernel_ptr() {
  return reinterpret_cast<const void*>(&chunk_gemm<Loop, kOutBf16, kProducer, kReduce>);
}

namespace {
struct Variant {
  InType in;
  bool out_bf16;
  bool producer;
  bool reduce;
  int bm, bn, bk;
  int threads;
  hipError_t (*launch)(const GemmArgs&, int32_t, hipStream_t, hipEvent_t, hipEvent_t);
  const void* (*func)();
};

#define CSG_VARIANT(IN, LOOP, OB, PR, RD)                                                                    \
  Variant {                                                                                                   \
    IN, OB, PR, RD, LOOP::BM, LOOP::BN, LOOP::BK, LOOP::THREADS, &launch_one<LOOP, OB, PR, RD>,               \
        &kernel_ptr<LOOP, OB, PR, RD>                                                                         \
  }

const Variant kVariants[] = {
    CSG_VARIANT(InType::BF16, LoopBf16_256, true, false, false),  CSG_VARIANT(InType::BF16, LoopBf16_256, true, true, false),
    CSG_VARIANT(InType::BF16, LoopBf16_256, false, false, false), CSG_VARIANT(InType::BF16, LoopBf16_256, false, true, false),
    CSG_VARIANT(InType::F32, LoopF32_64, false, false, false),    CSG_VARIANT(InType::F32, LoopF32_64, false, true, false),
    // GEMM + all-reduce: producers with the fused reduction
    CSG_VARIANT(InType::BF16, LoopBf16_256, true, true, true),    CSG_VARIANT(InType::BF16, LoopBf16_256, false, true, true),
    CSG_VARIANT(InType::F32, LoopF32_64, false, true, true),
    // smaller bf16 tiles for the consumers (more, shorter tiles: a chunk's tiles finish
    // sooner after it lands)
    CSG_VARIANT(InType::BF16, LoopBf16_256x128, true, false, false),
    CSG_VARIANT(InType::BF16, LoopBf16_128x256, true, false, false),
    CSG_VARIANT(InType::BF16, LoopBf16_128, true, false, false),
    // 128 x 256 for GEMM + reduce-scatter too: twice the tiles, so the emitted chunks
    // complete over more waves and fewer are left to copy after the last one
    CSG_VARIANT(InType::BF16, LoopBf16_128x256, true, true, false),
    // 256 x 224 tiles: N = 7 x 256 and 14 x 256 shapes fill every CU in whole waves
    CSG_VARIANT(InType::BF16, LoopBf16_256x224, true, false, false),
    CSG_VARIANT(InType::BF16, LoopBf16_256x224, false, false, false),
};

const Variant* find_variant(const KernelKey& k) {
  for (const Variant& v : kVariants)
    if (v.in == k.in && v.out_bf16 == k.out_bf16 && v.producer == k.producer && v.reduce == k.reduce &&
        v.bm == k.bm && v.bn == k.bn && v.bk == k.bk)
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
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, v->func(), v->threads, 0);
  if (e != hipSuccess) return e;
  if (per_cu < 1) per_cu = 1;
  *grid = cus * per_cu;
  return hipSuccess;
}

hipError_t launch_chunk_gemm(const KernelKey& key, const GemmArgs& args, int32_t grid, hipStream_t stream,
                             hipEvent_t start, hipEvent_t stop) {
  const Variant* v = find_variant(key);
  if (!v) return hipErrorInvalidValue;
  return v->launch(args, grid, stream, start, stop);
}

hipError_t launch_prologue(const PrologueArgs& args, hipStream_t stream) {
  hipLaunchKernelGGL(chunk_prologue, dim3(1), dim3(kPrologueThreads), 0, stream, args);
  return hipGetLastError();
}

}  // namespace csg
