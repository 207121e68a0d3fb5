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
// Both tiles reach LDS by DMA (buffer_load ... lds, no register staging) and stay
// unpadded: the K tile's 16-byte pieces and the V tile's 32-byte units are placed by XOR
// swizzles of the row index, and V^T fragments come from transposing reads
// (ds_read_b64_tr_b16), so the fragment reads are free of bank conflicts. The loop is
// software-pipelined by one block: on a chunk's last block the scores of the next block
// are computed from the other K buffer and discarded, one score block (16 MFMAs per
// wave) per chunk and unit. Scores are scaled into base 2 (exp2), and the log-sum-exp
// is returned in natural log.
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
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef short i16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef __attribute__((address_space(3))) unsigned char lds_u8_t;
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;

constexpr int D = kAttnHeadDim;
constexpr int BQ = kAttnBlockQ;
constexpr int BKV = kAttnBlockKV;
constexpr int kThreads = 256;         // 4 waves x 32 query rows
constexpr int kTileBytes = BKV * D * 2;   // one K or V tile: 16 KiB
constexpr int kBufferDword3 = 0x00020000;  // raw buffer resource word 3 (gfx9 family)
__device__ const bf16x2_t kBf16Ones = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
constexpr int kMaxAttnChunks = 4096;  // per-workgroup ready cache: one bit per chunk
constexpr float kLn2 = 0.6931471805599453f;
// Largest row sum of one block's weights accepted against the running reference; a
// larger (or non-finite) sum moves the reference to the row's maximum instead.
constexpr float kRowSumLimit = 65536.0f;

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

// K tile layout in LDS. Key row R (0..63) of the block has 16 pieces of 16 bytes (8
// head dims each); logical piece p sits in 16-byte slot
//     256 (p / 4) + 4 R + ((p % 4) ^ f(R)),   f(R) = ((R >> 2) ^ (R >> 1)) & 3.
// One DMA instruction fills 64 consecutive slots, i.e. one group of four pieces for 16
// rows, reading 64 contiguous bytes per row. A fragment read (16 consecutive rows, one
// logical piece) touches 16 distinct 16-byte bank groups, and any 8 aligned consecutive
// rows 8 distinct ones, so it is free of conflicts with 32 or 64 banks; and the slot's
// dependence on the piece index is an additive constant plus a bit that only depends on
// the piece's parity, so fragment reads use immediate offsets.
__device__ __forceinline__ int k_swz(int r) { return ((r >> 2) ^ (r >> 1)) & 3; }

// Buffer resource over [base, base + bytes) (bytes < 2^31), built from workgroup-
// uniform values so that it lives in SGPRs.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int bytes) {
  const uint64_t p = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(p));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(p >> 32));
  void* ub = reinterpret_cast<void*>((static_cast<uint64_t>(hi) << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(ub, 0, __builtin_amdgcn_readfirstlane(bytes), kBufferDword3);
}

// V tile layout in LDS: row-major, key row R (0..63) of 256 bytes, in which the 32-byte
// unit u (head dims 16 u .. + 15) sits at unit u ^ s(R % 4), s(q) = 2 q + q / 2. The
// value product reads V^T fragments with ds_read_b64_tr_b16, which transposes 4 x 16
// blocks among each 16 lanes: lane j of the 16 supplies the address of 4 consecutive
// elements, and lane i receives element i % 4 of lane 4 e + i / 4 as its element e.
// With lane j pointing at key k0 + j / 4, head dims d0 + 4 (j % 4), lane i receives
// head dim d0 + i of keys k0 .. k0 + 3. One such read touches 4 consecutive keys (R % 4
// = 0..3) x 16 or 32 dims, which the swizzle spreads over distinct bank groups with 32
// or 64 banks; the DMA writes rows contiguously as the K tile's does.
__device__ __forceinline__ int v_swz(int q) { return 2 * q + (q >> 1); }

// One 64-row block of key/value head g (rows [kv0, kv0 + 64) of the [rows][Hkv][D]
// array src) into a K or V tile at LDS byte address lds_tile, by LDS DMA: wave w fills
// LDS bytes 4096 w .. + 4095 with four 16-byte-per-lane loads of 1 KiB each. The tile
// layouts make the lane's source offset voff0 plus q times a fixed step (step_bytes):
// for K, instruction q covers rows 16 q .. + 15 (piece group w); for V, rows 16 w +
// 4 q .. + 3. The whole offset sits in the VGPR operand, which the buffer range check
// covers; the resource spans exactly the block's 64 rows of head g. Issued as inline asm
// (M0 saved and restored) so that the compiler does not wait for it before every LDS
// read: completion is waited for explicitly (wait_vm_all) before the barrier that
// publishes the tile.
__device__ __forceinline__ void dma_tile(const uint16_t* src, int hkv, int g, int kv0, uint32_t lds_tile, int wave,
                                         int voff0, int step_bytes) {
  const int64_t row = static_cast<int64_t>(hkv) * D;  // elements between consecutive keys
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(src + static_cast<int64_t>(kv0) * row + static_cast<int64_t>(g) * D,
                                              static_cast<int>(((BKV - 1) * row + D) * 2));
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane(lds_tile + 4096u * static_cast<uint32_t>(wave));
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint32_t saved;
    int voff;
    asm volatile(
        "v_add_u32 %1, %3, %4\n\t"
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %2\n\t"
        "buffer_load_dwordx4 %1, %5, 0 offen lds\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved), "=&v"(voff)
        : "s"(lds0 + 1024u * q), "s"(q * step_bytes), "v"(voff0), "s"(rs)
        : "memory");
  }
}

__device__ __forceinline__ void wait_vm_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Next work unit for a workgroup on die xcd (thread 0 only). The unit list, ordered by
// key/value head, is split into kXcdLists contiguous ranges, one per die, so that the
// units running on a die share key/value heads and stream the same key/value blocks
// through that die's L2 (with 8 key/value heads, one head per die). A die whose range
// is exhausted takes from the following dies' ranges; n_units when none has any left.
__device__ int next_unit(const AttnArgs& a, uint32_t xcd) {
  for (int d = 0; d < kXcdLists; ++d) {
    const int x = static_cast<int>((xcd + d) % kXcdLists);
    const int b0 = static_cast<int>(static_cast<int64_t>(a.n_units) * x / kXcdLists);
    const int len = static_cast<int>(static_cast<int64_t>(a.n_units) * (x + 1) / kXcdLists) - b0;
    if (len <= 0) continue;
    if (__hip_atomic_load(a.ticket + x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= static_cast<uint32_t>(len))
      continue;
    const uint32_t t = atomicAdd(a.ticket + x, 1u);
    if (t < static_cast<uint32_t>(len)) return b0 + static_cast<int>(t);
  }
  return a.n_units;
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

// S^T of one block of 64 keys (two 32-key tiles) for the wave's 32 query rows: lane
// (l32, hlf) ends with the scores of query row l32 against keys 32 kb + 8 (r / 4) +
// 4 hlf + r % 4 in sc[kb][r]. The lane's first operand is row 32 kb + l32, piece
// 2 s + hlf of the K tile: byte 4096 (s / 2) + 2048 kb + 64 l32 + 16 ((2 (s % 2) + hlf)
// ^ f(l32)); kEven / kOdd are the lane's part of it for even and odd s.
__device__ __forceinline__ void score_block(const unsigned char* kEven, const unsigned char* kOdd,
                                            const bf16x8_t (&qf)[D / 16], f32x16_t (&sc)[2]) {
  sc[0] = f32x16_t{};
  sc[1] = f32x16_t{};
#pragma unroll
  for (int s = 0; s < D / 16; ++s)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const unsigned char* p = ((s & 1) ? kOdd : kEven) + 4096 * (s >> 1) + 2048 * kb;
      const bf16x8_t kf = *reinterpret_cast<const bf16x8_t*>(p);
      sc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[s], sc[kb], 0, 0, 0);
    }
}

// Weights of one block against the reference m: exp2(scale_log2 s - m), packed to bf16
// in the second-operand order of the value product (step t takes registers
// 8 (t % 2) .. + 7 of tile t / 2, keys (t / 2) 32 + (t % 2) 16 + {4 hlf + 0..3,
// 8 + 4 hlf + 0..3}). Returns this lane's sum of the packed (bf16) weights, so that the
// normaliser adds up exactly the weights that the value product multiplies.
__device__ __forceinline__ float block_weights(const f32x16_t (&sc)[2], float scale_log2, float m,
                                               bf16x8_t (&pb)[4]) {
  float psum = 0.0f;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int kb = t >> 1, o = 8 * (t & 1);
    f32x8_t w;
#pragma unroll
    for (int r = 0; r < 8; ++r) w[r] = __builtin_amdgcn_exp2f(fmaf(sc[kb][o + r], scale_log2, -m));
    pb[t] = __builtin_convertvector(w, bf16x8_t);
    const bf16x2_t* pairs = reinterpret_cast<const bf16x2_t*>(&pb[t]);
#pragma unroll
    for (int i = 0; i < 4; ++i) psum = __builtin_amdgcn_fdot2_f32_bf16(pairs[i], kBf16Ones, psum, false);
  }
  return psum;
}

// Online softmax of one block. The running reference m of a query row moves only when
// it must: the block's weights are first taken against the current m, and only if the
// row's sum of them exceeds kRowSumLimit (or is not finite, as on a unit's first block,
// where m is -inf) does m move to the row's maximum scaled score, with the weights
// recomputed and the running sums rescaled. Both lanes of a row (lane and lane ^ 32)
// see the same row sum and the same maximum, so they keep the same m. The rare path is
// taken by the whole wave (with unchanged m on rows that do not need it), so its
// cross-lane exchange runs with every lane active. Returns the factor by which the
// accumulators are to be multiplied (1: unchanged); l is this lane's partial sum.
__device__ __forceinline__ float softmax_block(const f32x16_t (&sc)[2], float scale_log2, float& m, float& l,
                                               bf16x8_t (&pb)[4], bool& rescale) {
  float psum = block_weights(sc, scale_log2, m, pb);
  const float row = sum_halves(psum);
  const bool move = !(row <= kRowSumLimit);
  float alpha = 1.0f;
  rescale = __builtin_amdgcn_ballot_w64(move) != 0;
  if (rescale) {
    float mx = -__builtin_inff();
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[kb][r]);
    mx = max_halves(mx) * scale_log2;  // the scale is positive
    const float m_new = move ? fmaxf(m, mx) : m;
    alpha = __builtin_amdgcn_exp2f(m - m_new);  // 0 on a unit's first block, 1 on unmoved rows
    m = m_new;
    l *= alpha;
    psum = block_weights(sc, scale_log2, m, pb);
  }
  l += psum;
  return alpha;
}

// O^T += V^T . P^T for one block. The first operand of step t, head-dim tile db, is
// V^T rows 32 db + l32, keys in pb[t]'s order: two transposing reads of 4 keys each
// (keys (t / 2) 32 + (t % 2) 16 + 4 hlf + 0..3, then + 8). vt is the V tile; v_lane[db]
// is the lane's byte offset in it for keys 4 hlf + (lane % 16) / 4 and head dims
// 32 db + 16 ((lane / 16) % 2) + 4 (lane % 4); a block of 8 keys is 2048 bytes.
__device__ __forceinline__ void value_block(const lds_u8_t* vt, const int (&v_lane)[D / 32], const bf16x8_t (&pb)[4],
                                            f32x16_t (&acc)[D / 32]) {
  bf16x8_t vf[2][D / 32];  // fragments of steps t and t + 1: the reads run a step ahead
  auto load = [&](bf16x8_t (&f)[D / 32], int t) {
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      const lds_u8_t* p = vt + v_lane[db] + 256 * (32 * (t >> 1) + 16 * (t & 1));
      const i16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)(p));
      const i16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)(p + 2048));
      f[db] = __builtin_bit_cast(bf16x8_t, (i16x8_t{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]}));
    }
  };
  load(vf[0], 0);
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    if (t + 1 < 4) load(vf[(t + 1) & 1], t + 1);
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
      acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[t & 1][db], pb[t], acc[db], 0, 0, 0);
  }
}

}  // namespace

__global__ __launch_bounds__(kThreads, 2) void ring_attn(AttnArgs a) {
  // K and V tiles, double-buffered
  __shared__ __attribute__((aligned(1024))) unsigned char sK[2 * kTileBytes];
  __shared__ __attribute__((aligned(1024))) unsigned char sV[2 * kTileBytes];
  __shared__ uint32_t ready_bits[kMaxAttnChunks / 32];
  __shared__ int s_unit;
  __shared__ int s_state;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, hlf = lane >> 5;
  // K tile: this lane's DMA source offset (row L / 4, piece 4 wave + ((L % 4) ^ f(row)),
  // 16 rows further per instruction) and its fragment-read offsets for even and odd
  // pieces. V tile: DMA source offset (row 16 wave + L / 16, unit ((L % 16) / 2) ^
  // s(row % 4), half L % 2; 4 rows further per instruction) and transposing-read
  // offsets per head-dim tile.
  const int key_bytes = a.Hkv * D * 2;
  const int k_voff0 = (lane >> 2) * key_bytes + (4 * wave + ((lane & 3) ^ k_swz(lane >> 2))) * 16;
  const int v_voff0 = (16 * wave + (lane >> 4)) * key_bytes + ((((lane & 15) >> 1) ^ v_swz(lane >> 4)) * 32) +
                      (lane & 1) * 16;
  const uint32_t sK_addr =
      __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_ptr_t)sK)));
  const uint32_t sV_addr =
      __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_ptr_t)sV)));
  const int k_even = 64 * l32 + 16 * (hlf ^ k_swz(l32));
  const int k_odd = 64 * l32 + 16 * ((2 + hlf) ^ k_swz(l32));
  int v_lane[D / 32];
  {
    const int i = lane & 15, h = (lane >> 4) & 1;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
      v_lane[db] = 256 * ((i >> 2) + 4 * hlf) + 32 * ((2 * db + h) ^ v_swz(i >> 2)) + 8 * (i & 3);
  }
  const lds_u8_t* sV_lds = (const lds_u8_t*)(sV);
  if (blockIdx.x == 0 && a.next_ticket) {
    // clear the next call's state set (its prologue, folded into this kernel)
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
  for (int i = tid; i < kMaxAttnChunks / 32; i += kThreads) ready_bits[i] = 0;
  uint32_t xcd;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID, 0, 4)" : "=s"(xcd));
  xcd %= kXcdLists;
  const int n_qb = (a.Sq + BQ - 1) / BQ;
  const int G = a.H / a.Hkv;
  uint32_t units = 0;

  for (;;) {
    __syncthreads();  // everyone is done with s_unit / s_state / LDS of the previous unit
    if (tid == 0) {
      int u = next_unit(a, xcd);
      if (load_flag(&a.diag->abort)) u = a.n_units;
      s_unit = u;
    }
    __syncthreads();
    const int u = __builtin_amdgcn_readfirstlane(s_unit);
    if (u >= a.n_units) break;
    ++units;
    // unit -> (key/value head g, query block, head of g's group): consecutive units, and
    // so a die's range of them, share key/value heads
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
      if (__builtin_amdgcn_readfirstlane(s_state) < 0) {
        aborted = true;
        break;
      }
      // Blocks j = 0 .. nb - 1 of the chunk, software-pipelined by one block: while the
      // matrix cores compute the scores of block j + 1, the vector unit computes the
      // softmax of block j (the two are independent). Tiles are DMA'd into LDS a step
      // ahead of use (K of block j + 2 and V of block j + 1 during step j) into double
      // buffers (K of block j in buffer j % 2, V likewise), so one barrier per block
      // publishes the step's tiles and frees the previous step's.
      const int r0 = a.chunk_rows[2 * c], r1 = a.chunk_rows[2 * c + 1];
      const int nb = (r1 - r0) / BKV;
      if (nb > 0) {
        dma_tile(a.K, a.Hkv, g, r0, sK_addr, wave, k_voff0, 16 * key_bytes);
        dma_tile(a.V, a.Hkv, g, r0, sV_addr, wave, v_voff0, 4 * key_bytes);
        if (nb > 1) dma_tile(a.K, a.Hkv, g, r0 + BKV, sK_addr + kTileBytes, wave, k_voff0, 16 * key_bytes);
        wait_vm_all();
        __syncthreads();
        // One step: block j's softmax and value product, block j + 1's scores. The scores
        // of the current and next block alternate between sa and sb (the loop runs two
        // steps per iteration), so no register copies are needed.
        auto step = [&](int j, const f32x16_t (&cur)[2], f32x16_t (&nxt)[2]) {
          const int kv0 = r0 + j * BKV;
          const int buf = j & 1, nbuf = buf ^ 1;
          wait_vm_all();    // this wave's parts of V j and K j + 1 have landed
          __syncthreads();  // ... everyone's; and everyone is done with K j and V j - 1
          if (j + 2 < nb)
            dma_tile(a.K, a.Hkv, g, kv0 + 2 * BKV, sK_addr + buf * kTileBytes, wave, k_voff0, 16 * key_bytes);
          if (j + 1 < nb)
            dma_tile(a.V, a.Hkv, g, kv0 + BKV, sV_addr + nbuf * kTileBytes, wave, v_voff0, 4 * key_bytes);
          // scores of block j + 1 (on the chunk's last block, of whatever the other
          // buffer holds: computed and discarded, which keeps this code branch-free so
          // that the compiler can interleave the two independent streams)
          score_block(sK + nbuf * kTileBytes + k_even, sK + nbuf * kTileBytes + k_odd, qf, nxt);
          bf16x8_t pb[4];
          bool rescale;
          const float alpha = softmax_block(cur, a.scale_log2, m, l, pb, rescale);
          if (rescale) {
#pragma unroll
            for (int db = 0; db < D / 32; ++db) acc[db] *= alpha;
          }
          value_block(sV_lds + buf * kTileBytes, v_lane, pb, acc);
        };
        f32x16_t sa[2], sb[2];
        score_block(sK + k_even, sK + k_odd, qf, sa);
        int j = 0;
        for (; j + 1 < nb; j += 2) {
          step(j, sa, sb);
          step(j + 1, sb, sa);
        }
        if (j < nb) step(j, sa, sb);
      }
      // every load of this chunk's rows that the workgroup uses has landed (each block's
      // loads are waited for before its LDS stores, and every thread has passed the
      // barrier after the chunk's last stores); prefetches still in flight re-read the
      // chunk's last block and are discarded
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
