// Device side of libpfxattn: kernels for gfx950 (CDNA4) and the entry points
// that launch them.
//
// Attention layout on the MFMA units (v_mfma_f32_16x16x32_bf16, wave64):
//   S^T = K Q^T     A = 16 keys x 32 head dims (one page of one KV head per
//                   tile), B = 32 head dims x 16 query columns; each lane
//                   ends up holding 4 scores of one query column.
//   O^T = V^T P^T   A = 16 head dims x 32 keys, B = 32 keys x 16 columns,
//                   taken straight from the lane's own scores, so the
//                   online-softmax statistics of a column never leave the
//                   four lanes that own it.
// V^T is read from the LDS stage with ds_read_b64_tr_b16, which hands each
// lane 4 keys of one head dim out of a key-major tile.
//
// Up to three launches per call, in stream order (a batch with both extend
// blocks and decode pieces runs the first two as one launch, the extend
// blocks leading its grid):
//   extend blocks: one workgroup per block of <= 128 query columns of one
//     request and one KV head, streaming the prefix and the causal suffix
//     through an LDS ring; rows written directly.
//   decode: one workgroup per piece, or persistent ones.  The decode items (an agent's prefix
//     against a block of its decode rows, a request's suffix against its own
//     rows; one KV head each) are cut into pieces of at most 64 32-key
//     steps, listed longest first and dealt to the workgroups in rounds; a
//     workgroup's pieces flow through one LDS ring without a break at piece
//     boundaries, and every piece leaves a partial state.
//   merge: every decode row combines its pieces' partial states by
//     log-sum-exp weights.
// The launch boundaries order the phases: no atomics or device-wide fences.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <mutex>
#include <type_traits>

#include "pfx_internal.h"

namespace pfx {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
// Lazy rescaling: the running maximum is only raised when a new score
// exceeds it by more than this (log2 units), so exp2 arguments stay <= 8.
constexpr float kRescaleSlack = 8.0f;
// Finite "minus infinity" for the running maximum: exp2(score - kNegBig) of a
// masked score (-inf) is still 0, and no inf - inf can arise.
constexpr float kNegBig = -1.0e30f;

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Four bf16 (two packed words, low element first) as floats.
__device__ __forceinline__ f32x4 unpack_bf16x4(uint32_t a, uint32_t b) {
  return f32x4{__builtin_bit_cast(float, a << 16), __builtin_bit_cast(float, a & 0xFFFF0000u),
               __builtin_bit_cast(float, b << 16), __builtin_bit_cast(float, b & 0xFFFF0000u)};
}

// A partial state's D values in the plan's workspace: the piece's
// accumulators divided by its own sum l (a convex combination of V rows, so
// within V's range), as bf16.  The G rows of one slot (one decode token
// against the G query heads of a KV head: rows r0 .. r0 + G - 1, r0 a
// multiple of G) fill the G * D elements from element r0 * D as 16-byte
// units, unit-major: unit u = 4 p + grp of row g holds dims 32 p + 4 grp
// .. + 3 and 32 p + 16 + 4 grp .. + 3 (two f32x4 of the MFMA accumulator
// layout, blocks 2 p and 2 p + 1) at element (u * G + g) * 8.  A wave's
// store of one unit then covers each token's G rows as one run of 64 G
// bytes.  The stores are non-temporal: whole lines that the merge launch
// reads once, not kept dirty in the L2 of the XCD that wrote them until the
// end of the launch.
// Unit grp of row `row` (query head g of its token); unit 4 p + grp is at
// that pointer + part_unit_stride(G) * p.
__device__ __forceinline__ uint16_t* part_unit0(uint16_t* o_part, size_t row, int g, int G, int grp, int D) {
  return o_part + (row - size_t(g)) * D + size_t(grp * G + g) * 8;
}
__device__ __forceinline__ int part_unit_stride(int G) { return 32 * G; }

// Store a lane's accumulators (dims 16 blk + 4 grp + i) as its units of a
// partial row, scaled by inv = 1 / l (0 for a piece that saw no key).
template <int D>
__device__ __forceinline__ void store_partial(uint16_t* o_part, size_t row, int g, int G, int grp,
                                              const f32x4 (&acc)[D / 16], float inv) {
  uint16_t* out = part_unit0(o_part, row, g, G, grp, D);
#pragma unroll
  for (int p = 0; p < D / 32; ++p) {
    const f32x4 x = acc[2 * p], y = acc[2 * p + 1];
    const u32x4 w = {pack_bf16(x[0] * inv, x[1] * inv), pack_bf16(x[2] * inv, x[3] * inv),
                     pack_bf16(y[0] * inv, y[1] * inv), pack_bf16(y[2] * inv, y[3] * inv)};
    __builtin_nontemporal_store(w, reinterpret_cast<u32x4*>(out + part_unit_stride(G) * p));
  }
}

// Placed inside a rarely taken branch (masking, rescaling): the compiler may
// not turn the branch into always-executed selects.
#define PFX_KEEP_BRANCH() asm volatile("" ::: "memory")

// Max / sum over the four lanes l, l ^ 16, l ^ 32, l ^ 48 (the lanes holding
// one query column), with the gfx950 row-swap instructions instead of LDS
// permutes.  v_permlane16_swap a, b exchanges the odd 16-lane rows of a with
// the even rows of b, v_permlane32_swap the upper half of a with the lower
// half of b; applied to two copies of x, the pair holds {own, partner} in
// every lane, so all four lanes end with the same value.  Issued through asm:
// the compiler's builtins for these instructions return the first register
// for both results.  The nops keep clear of VALU-to-permlane hazards.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void row_swap16(uint32_t& a, uint32_t& b) {
  asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1\n\ts_nop 1" : "+v"(a), "+v"(b));
}
__device__ __forceinline__ void row_swap32(uint32_t& a, uint32_t& b) {
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 1" : "+v"(a), "+v"(b));
}
#pragma clang diagnostic pop

__device__ __forceinline__ float column_max(float x) {
  uint32_t a = __builtin_bit_cast(uint32_t, x), b = a;
  row_swap16(a, b);
  x = __builtin_elementwise_maximum(__builtin_bit_cast(float, a), __builtin_bit_cast(float, b));
  a = __builtin_bit_cast(uint32_t, x);
  b = a;
  row_swap32(a, b);
  return __builtin_elementwise_maximum(__builtin_bit_cast(float, a), __builtin_bit_cast(float, b));
}
__device__ __forceinline__ float column_sum(float x) {
  uint32_t a = __builtin_bit_cast(uint32_t, x), b = a;
  row_swap16(a, b);
  x = __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b);
  a = __builtin_bit_cast(uint32_t, x);
  b = a;
  row_swap32(a, b);
  return __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b);
}

struct AttnArgs {
  const uint16_t* kpool;
  const uint16_t* vpool;
  const uint16_t* q;
  uint16_t* o;
  float* lse;
  DevPlan plan;
  int32_t hq, hkv, group, group_shift;
  int32_t num_workers;  // decode launch: persistent workgroups
  int32_t num_pieces;   // decode pieces in the plan
  float scale_log2;  // sm_scale * log2(e)
  // Decode with the KV append folded in: a suffix piece takes its new
  // tokens' K/V rows straight from k_new / v_new (rows [T][Hkv][D], token
  // order) and the merge launch writes them into the pool.  fuse_append ==
  // 0: the append ran before the launch and the pool already holds them.
  const uint16_t* k_new;
  const uint16_t* v_new;
  int32_t fuse_append;
  // Decode launch: its first num_wide workgroups run the wide prefix blocks
  // items[wide_first ...], the others the decode pieces.
  int32_t num_wide, wide_first;
  // Merge launch: P when every (merge row m, KV head h) has P parts from
  // slot (m Hkv + h) P (then merge_head is not read), else 0; and 1 when
  // merge row m is token m for every m (then the merge with the append
  // folded in reads no merge_tok: the append's chain of loads, merge_tok,
  // then tok_slot and the new rows, loses a round trip.  Without the
  // append the load stays: measured, skipping it there was no faster).
  int32_t merge_parts, merge_tok_is_row;
};

// Geometry of one 32-key step of an item.
struct StepPos {
  int32_t list_off;      // offset of the segment's page list in the plan's page list
  int32_t k0, kend;      // first key of the step, end of the segment
  int32_t seg;           // 0: prefix (no mask), 1: suffix (causal)
};

__device__ __forceinline__ StepPos step_pos(const Item& it, int st, int s0_steps) {
  StepPos p;
  if (st < s0_steps) {
    p.list_off = it.s0_page_off;
    p.k0 = it.s0_kbeg + st * kStepKeys;
    p.kend = it.s0_kend;
    p.seg = 0;
  } else {
    p.list_off = it.s1_page_off;
    p.k0 = it.s1_kbeg + (st - s0_steps) * kStepKeys;
    p.kend = it.s1_kend;
    p.seg = 1;
  }
  return p;
}

// The steps of an extend block where the common path changes, found once
// per block so that an ordinary step needs no position arithmetic:
//   tail0, tail1: the last step of segment 0 / 1 when the segment ends
//     inside it (keys to mask, V to zero), else -1;
//   half0, half1: such a step when its second page does not exist, else -1;
//   diag: the first suffix step with a key past the wave's lowest limit
//     (from there on every suffix step is masked);
//   d1: page-table index of step st's first page is 2 st, plus d1 in
//     segment 1.
struct StepMarks {
  int32_t s0_steps, nsteps, d1, tail0, tail1, half0, half1, diag;
};

__device__ __forceinline__ StepMarks step_marks(const Item& it, int p0n, int lim_lo) {
  StepMarks mk;
  const int s0_steps = (it.s0_kend - it.s0_kbeg + kStepKeys - 1) / kStepKeys;
  const int s1_steps = (it.s1_kend - it.s1_kbeg + kStepKeys - 1) / kStepKeys;
  mk.s0_steps = s0_steps;
  mk.nsteps = s0_steps + s1_steps;
  mk.d1 = p0n - 2 * s0_steps;
  const int last0 = it.s0_kbeg + kStepKeys * (s0_steps - 1);  // first key of segment 0's last step
  const int last1 = it.s1_kbeg + kStepKeys * (s1_steps - 1);
  mk.tail0 = s0_steps > 0 && last0 + kStepKeys > it.s0_kend ? s0_steps - 1 : -1;
  mk.half0 = s0_steps > 0 && last0 + 16 >= it.s0_kend ? s0_steps - 1 : -1;
  mk.tail1 = s1_steps > 0 && last1 + kStepKeys > it.s1_kend ? mk.nsteps - 1 : -1;
  mk.half1 = s1_steps > 0 && last1 + 16 >= it.s1_kend ? mk.nsteps - 1 : -1;
  // Suffix step j is masked once its last key s1_kbeg + 32 j + 31 passes lim_lo.
  const int x = lim_lo - it.s1_kbeg - (kStepKeys - 1);
  mk.diag = s1_steps == 0 ? 0x7fffffff : s0_steps + (x < 0 ? 0 : x / kStepKeys + 1);
  return mk;
}

template <int D, int QB>
struct WaveState {
  static constexpr int CH = D / 16;
  f32x4 acc[QB][CH];  // O^T: lane holds dims 16 blk + 4 grp + i of its column, [blk][i]
  float m[QB];        // running max (log2 units), same in the 4 lanes of a column
  f32x4 lv[QB];       // running sum from the matrix unit: element 0 in the group-0 lanes, 0 elsewhere
};

template <int D, int QB>
__device__ __forceinline__ void reset_state(WaveState<D, QB>& ws) {
#pragma unroll
  for (int b = 0; b < QB; ++b) {
    ws.m[b] = kNegBig;
    ws.lv[b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int jj = 0; jj < D / 16; ++jj) ws.acc[b][jj] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
}

// Merge `nparts` partial results for 8 consecutive dims of one row:
//   lse = ln sum_k exp(lse_k),  O = sum_k exp(lse_k - lse) O_k.
// o_row points at dims d0..d0+7 of partial 0; partial k is o_stride floats
// further on; lse_k is at l_row[k * l_stride].
__device__ __forceinline__ void merge_row8(const float* o_row, size_t o_stride, const float* l_row, size_t l_stride,
                                           int nparts, uint16_t* out8, float* lse_out) {
  float mx = -INFINITY;
  for (int k = 0; k < nparts; ++k) mx = fmaxf(mx, l_row[k * l_stride]);
  float z = 0.f;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int k = 0; k < nparts; ++k) {
    const float w = fast_exp2((l_row[k * l_stride] - mx) * kLog2e);
    z += w;
    const f32x4 a = *reinterpret_cast<const f32x4*>(o_row + k * o_stride);
    const f32x4 b = *reinterpret_cast<const f32x4*>(o_row + k * o_stride + 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[e] += w * a[e];
      acc[4 + e] += w * b[e];
    }
  }
  const float inv = 1.0f / z;
  u32x4 ow;
#pragma unroll
  for (int e = 0; e < 4; ++e) ow[e] = pack_bf16(acc[2 * e] * inv, acc[2 * e + 1] * inv);
  *reinterpret_cast<u32x4*>(out8) = ow;
  if (lse_out) *lse_out = mx + logf(z);
}

// ---------------------------------------------------------------------------
// LDS-staged K/V shared by the four waves of a workgroup.
//
// A step's K/V (two 16-token pages of one KV head, K and V) is copied from
// the pool straight into LDS with global_load_lds_dwordx4 -- no registers
// involved -- through a ring of kStages buffers, so kStages - 1 steps are in
// flight while one is consumed.  Each wave loads one quarter of a step (one
// page of K or of V) and consumes all of it for its own query columns; a
// barrier per step publishes the stage and frees the one to be refilled.
// Inside a page tile the 16-byte chunk c of token t sits at slot
// t * chunks + (c ^ t): the MFMA operand reads (16 tokens at one chunk, or
// one token's 16 chunks) then fall in 16 different bank groups.
// ---------------------------------------------------------------------------
// Stages of the LDS ring: three in flight while one is consumed.
constexpr int kStages = 4;

template <int D>
struct TileGeom {
  static constexpr int chunks = D / 8;                 // 16-byte chunks per token row
  static constexpr int page_bytes = 16 * D * 2;        // one (page, KV head) block
  static constexpr int stage_bytes = 4 * page_bytes;   // K tile 0, K tile 1, V tile 0, V tile 1
  static constexpr int loads_per_wave = page_bytes / 1024;
};

// Chunk c of token row t sits at slot t * chunks + (c ^ row_key(t)).  LDS
// on gfx950 has 64 banks of 4 bytes (a 256-byte period).  A 16-byte read is
// served in four cycles of 16 lanes each: four blocks of four consecutive
// lanes, the blocks of one half-wave split by the parity of the low three
// bits of their index (lanes 0-3, 12-15, 20-27 together).  An 8-byte read,
// plain or transposing, is served in two cycles of 32 consecutive lanes.
// (Both measured with the bank-conflict counter on in-bounds probes.)  For
// 256-byte rows the key below is an XOR-linear map (bits 0..3 of t to 2, 4,
// 13, 8) chosen so that the three read patterns here see no conflict: the K
// operand reads (lane (col, grp): row col, chunk 4 s + grp), the row reads
// of V (row 4 grp + i, chunk col) and the transposing V reads (row
// 4 grp + e, chunks 2 blk and 2 blk + 1).  For 128-byte rows no XOR key
// clears all three; this one leaves the transposing reads free.
template <int chunks>
__device__ __forceinline__ int row_key(int t) {
  if constexpr (chunks == 16) return ((t & 3) << 1) ^ (t & 8) ^ (-((t >> 2) & 1) & 13);
  else return (((t >> 1) & 3) << 1) | ((t >> 3) & 1);
}
template <int chunks>
__device__ __forceinline__ int swizzled_slot(int t, int c) { return t * chunks + (c ^ row_key<chunks>(t)); }

// Byte offsets, within a (page, KV head) block, of the chunk that this lane
// copies into slot 64 j + lane of the swizzled layout, less 1024 j (slot
// 64 j + lane is row t = 64 j / chunks + lane / chunks, so the rows of copy j
// start 1024 j bytes in).
template <int D>
__device__ __forceinline__ void block_lane_offsets(uint32_t (&off)[TileGeom<D>::loads_per_wave], int lane) {
  using TG = TileGeom<D>;
#pragma unroll
  for (int j = 0; j < TG::loads_per_wave; ++j) {
    const int t = (64 * j + lane) / TG::chunks;
    const int c = (lane % TG::chunks) ^ row_key<TG::chunks>(t);
    off[j] = uint32_t(2 * (t * D + 8 * c) - 1024 * j);
  }
}

// Wait until at most n of this wave's vector-memory operations are pending.
__device__ __forceinline__ void wait_vmcnt(int n) {
  // s_waitcnt encoding on gfx9: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] at [15:14].
#define PFX_VMCNT(N) __builtin_amdgcn_s_waitcnt(((N) & 15) | (7 << 4) | (15 << 8) | (((N) >> 4) << 14))
  switch (n) {
    case 0: PFX_VMCNT(0); break;
    case 1: PFX_VMCNT(1); break;
    case 2: PFX_VMCNT(2); break;
    case 3: PFX_VMCNT(3); break;
    case 4: PFX_VMCNT(4); break;
    case 5: PFX_VMCNT(5); break;
    case 6: PFX_VMCNT(6); break;
    case 7: PFX_VMCNT(7); break;
    case 8: PFX_VMCNT(8); break;
    case 9: PFX_VMCNT(9); break;
    case 10: PFX_VMCNT(10); break;
    case 11: PFX_VMCNT(11); break;
    case 12: PFX_VMCNT(12); break;
    case 13: PFX_VMCNT(13); break;
    case 14: PFX_VMCNT(14); break;
    case 15: PFX_VMCNT(15); break;
    case 16: PFX_VMCNT(16); break;
    case 17: PFX_VMCNT(17); break;
    case 18: PFX_VMCNT(18); break;
    case 19: PFX_VMCNT(19); break;
    case 20: PFX_VMCNT(20); break;
    case 21: PFX_VMCNT(21); break;
    case 22: PFX_VMCNT(22); break;
    case 23: PFX_VMCNT(23); break;
    case 24: PFX_VMCNT(24); break;
    case 25: PFX_VMCNT(25); break;
    case 26: PFX_VMCNT(26); break;
    case 27: PFX_VMCNT(27); break;
    case 28: PFX_VMCNT(28); break;
    case 29: PFX_VMCNT(29); break;
    case 30: PFX_VMCNT(30); break;
    case 31: PFX_VMCNT(31); break;
    default: PFX_VMCNT(32); break;
  }
#undef PFX_VMCNT
}

typedef __attribute__((address_space(3))) unsigned char* lds_bytes;

// Copy 16 bytes per lane from global memory into LDS at lds_addr + 16 * lane
// (global_load_lds_dwordx4; M0 holds the wave-uniform LDS address).  Issued
// through asm so the compiler's wait insertion does not treat every later
// LDS read as dependent on every copy in flight: completion is awaited
// explicitly with wait_vmcnt before the barrier that publishes a stage.
// M0 is otherwise unused by these kernels (tests/test_build_checks.py checks
// the generated code for that).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void copy16_to_lds(const void* src, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(lds_addr) : "memory", "m0");
}

// Copy one wave's share of a (page, KV head) block, L KiB, into LDS at
// lds_addr: copy j reads base + off[j] + 1024 j and writes
// lds_addr + 1024 j + 16 * lane.  The base is wave-uniform and goes in
// SGPRs; the instruction offset 1024 j moves both the global and the LDS
// address, so one M0 serves all L copies and the lane offsets are computed
// once per block.
template <int L>
__device__ __forceinline__ void copy_block_to_lds(const void* base, const uint32_t (&off)[L], uint32_t lds_addr) {
  static_assert(L == 2 || L == 4, "a block is 2 or 4 KiB");
  const uint64_t b = reinterpret_cast<uintptr_t>(base);
  // readfirstlane yields an int: take each half as unsigned before joining.
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(uint32_t(b))));
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(uint32_t(b >> 32))));
  const uint64_t sb = (uint64_t(hi) << 32) | lo;
  const uint32_t m = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(lds_addr)));
  if constexpr (L == 4)
    asm volatile(
        "s_mov_b32 m0, %1\n\t"
        "global_load_lds_dwordx4 %2, %0\n\t"
        "global_load_lds_dwordx4 %3, %0 offset:1024\n\t"
        "global_load_lds_dwordx4 %4, %0 offset:2048\n\t"
        "global_load_lds_dwordx4 %5, %0 offset:3072" ::"s"(sb),
        "s"(m), "v"(off[0]), "v"(off[1]), "v"(off[2]), "v"(off[3])
        : "memory", "m0");
  else
    asm volatile(
        "s_mov_b32 m0, %1\n\t"
        "global_load_lds_dwordx4 %2, %0\n\t"
        "global_load_lds_dwordx4 %3, %0 offset:1024" ::"s"(sb),
        "s"(m), "v"(off[0]), "v"(off[1])
        : "memory", "m0");
}
#pragma clang diagnostic pop

__device__ __forceinline__ uint32_t lds_address(const unsigned char* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_bytes)(p)));
}


typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) s16x4* lds_s16x4;

// V^T operand of output block blk (dims 16 blk .. 16 blk + 15 as the MFMA
// rows) for the step's 32 keys in score order (tile 0 keys 4 grp + e, then
// tile 1 keys 4 grp + e): two ds_read_b64_tr_b16.  Within a 16-lane group
// that instruction hands output lane i element e of what input lane
// 4 e + i / 4 addressed, element i % 4; so lane 4 e + q addresses key
// 4 grp + e, dims 16 blk + 4 q .. + 3, and lane i receives dim 16 blk + i
// of the four keys.
template <int D>
__device__ __forceinline__ bf16x8 v_operand_tr(const unsigned char* v0, const unsigned char* v1, int blk, int lane) {
  constexpr int chunks = D / 8;
  const int s = lane & 15;
  const int row = 4 * (lane >> 4) + (s >> 2);
  const int q = s & 3;
  const int off = 16 * swizzled_slot<chunks>(row, 2 * blk + (q >> 1)) + 8 * (q & 1);
  const s16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4)(v0 + off));
  const s16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4)(v1 + off));
  // Concatenated as 16-bit vectors: through 32-bit words, the compiler
  // rebuilds the bf16 elements with a bitfield insert per register.
  const s16x8 ab = __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, ab);
}

// Zero, in a step's V^T operands, the keys at or past kend (their slots may
// hold anything, and 0 * NaN is NaN).  Element e of each half of an operand
// is key k0 + 16 t + 4 grp + e.
// The masks are applied by an opaque AND: written as C, the compiler folds
// them into bitfield inserts that it then also runs, as no-ops, on the steps
// that need no zeroing.
__device__ __forceinline__ uint32_t and_opaque(uint32_t x, uint32_t m) {
  uint32_t r;
  asm volatile("v_and_b32 %0, %1, %2" : "=v"(r) : "v"(x), "v"(m));
  return r;
}
template <int D>
__device__ __forceinline__ void zero_v_tail(bf16x8 (&vop)[D / 16], int k0, int kend, int grp) {
  uint32_t keep[2][2];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
      const int key = k0 + 16 * t + 4 * grp + 2 * h2;  // element 2 h2 (low half) and 2 h2 + 1 (high half)
      keep[t][h2] = (key < kend ? 0x0000FFFFu : 0u) | (key + 1 < kend ? 0xFFFF0000u : 0u);
    }
#pragma unroll
  for (int blk = 0; blk < D / 16; ++blk) {
    u32x4 w = __builtin_bit_cast(u32x4, vop[blk]);
    w[0] = and_opaque(w[0], keep[0][0]);
    w[1] = and_opaque(w[1], keep[0][1]);
    w[2] = and_opaque(w[2], keep[1][0]);
    w[3] = and_opaque(w[3], keep[1][1]);
    vop[blk] = __builtin_bit_cast(bf16x8, w);
  }
}

// One 32-key step (two 16-key pages staged in LDS: K tile 0, K tile 1,
// V tile 0, V tile 1) against the wave's QB blocks of 16 query columns
// (the first nblk of them in use):
//   S^T = K Q^T: lane (col, grp) gets the scores of keys 16 t + 4 grp + i;
//   online softmax in log2 units, the running maximum raised lazily;
//   O^T += V^T P^T with P straight from the lane's own scores.
// Keys at or past kend, and (causal) keys past a column's limit, are masked.
template <int D, int QB>
__device__ __forceinline__ void attend_step(WaveState<D, QB>& ws, const unsigned char* stage,
                                            const bf16x8 (&qf)[QB][D / 32], const int (&lim)[QB], int k0,
                                            int kend, bool causal, int nblk, int lane, float scale_log2) {
  using TG = TileGeom<D>;
  constexpr int KS = D / 32;
  constexpr int CH = D / 16;
  const int col = lane & 15, grp = lane >> 4;
  const bool tail = k0 + kStepKeys > kend;
  f32x4 sc[QB][2];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    u32x4 kf[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s)
      kf[s] = *reinterpret_cast<const u32x4*>(stage + t * TG::page_bytes +
                                              16 * swizzled_slot<TG::chunks>(col, 4 * s + grp));
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      if (b >= nblk) break;
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < KS; ++s)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kf[s]), qf[b][s], acc, 0, 0, 0);
      sc[b][t] = acc;
    }
  }
  bf16x8 pb[QB];
#pragma unroll
  for (int b = 0; b < QB; ++b) {
    if (b >= nblk) break;
    float v[8] = {sc[b][0][0], sc[b][0][1], sc[b][0][2], sc[b][0][3], sc[b][1][0], sc[b][1][1], sc[b][1][2], sc[b][1][3]};
    if (tail || causal) {
      PFX_KEEP_BRANCH();
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = k0 + 16 * t + 4 * grp + i;
          if (key >= kend || (causal && key > lim[b])) v[4 * t + i] = -INFINITY;
        }
    }
    float x[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = v[i];
#pragma unroll
    for (int w = 4; w >= 1; w /= 2)
#pragma unroll
      for (int i = 0; i < w; ++i) x[i] = __builtin_elementwise_maximum(x[i], x[i + w]);
    float mx = x[0];  // IEEE maximum: no NaN canonicalisation of the MFMA results
    // The cross-lane max is needed only when some lane passes m + slack.
    if (__any(mx * scale_log2 > ws.m[b] + kRescaleSlack)) {
      PFX_KEEP_BRANCH();
      mx = column_max(mx) * scale_log2;  // scale > 0: max of the scaled scores
      const bool raise = mx > ws.m[b] + kRescaleSlack;
      const float mnew = raise ? mx : ws.m[b];
      const float alpha = fast_exp2(ws.m[b] - mnew);
      ws.lv[b][0] *= alpha;  // rows other than 0 stay zero
#pragma unroll
      for (int jj = 0; jj < CH; ++jj) ws.acc[b][jj] *= alpha;
      ws.m[b] = mnew;
    }
    const float neg_m = -ws.m[b];
    float pr[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) pr[j] = fast_exp2(fmaf(v[j], scale_log2, neg_m));
    u32x4 pw = {pack_bf16(pr[0], pr[1]), pack_bf16(pr[2], pr[3]), pack_bf16(pr[4], pr[5]), pack_bf16(pr[6], pr[7])};
    pb[b] = __builtin_bit_cast(bf16x8, pw);
  }
  bf16x8 vop[CH];
#pragma unroll
  for (int blk = 0; blk < CH; ++blk)
    vop[blk] = v_operand_tr<D>(stage + 2 * TG::page_bytes, stage + 3 * TG::page_bytes, blk, lane);
  if (tail) {
    PFX_KEEP_BRANCH();
    zero_v_tail<D>(vop, k0, kend, grp);
  }
#pragma unroll
  for (int blk = 0; blk < CH; ++blk) {
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      if (b >= nblk) break;
      ws.acc[b][blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop[blk], pb[b], ws.acc[b][blk], 0, 0, 0);
    }
  }
  // Row sums of P on the matrix unit (row 0 of the A operand is ones).
  const uint32_t one2 = col == 0 ? 0x3F803F80u : 0u;
  const bf16x8 ones_row0 = __builtin_bit_cast(bf16x8, u32x4{one2, one2, one2, one2});
#pragma unroll
  for (int b = 0; b < QB; ++b) {
    if (b >= nblk) break;
    ws.lv[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones_row0, pb[b], ws.lv[b], 0, 0, 0);
  }
}

// ---------------------------------------------------------------------------
// Decode on the vector ALU (a plan option): the same pieces, LDS ring and
// online softmax as above, with both contractions done by two-wide bf16 dot
// products (v_dot2_f32_bf16) instead of the matrix unit.  It exists to set
// the two engines side by side on counters; the matrix unit is the default.
//
// Scores: lane (col, grp) holds its column's whole Q row and forms the
// scores of keys 16 t + 4 grp + i, the MFMA layout, so masking and the
// softmax are the same code.
// P V: lane (c, grp) accumulates columns 4 grp .. 4 grp + 3 at dims
// 16 blk + c over all 32 keys of a step.  V^T comes from the transposing LDS
// read (two keys per word, as the MFMA path reads it, for all four key
// groups), P from an exchange through LDS (each lane publishes the packed P
// of its column and keys).  At the end of a piece the accumulators are
// transposed into the MFMA state layout through LDS.
// All exchanges stay inside one wave: LDS serves a wave's instructions in
// order, and a wave-scope fence keeps the compiler from reordering them.
// ---------------------------------------------------------------------------
// LDS per wave: P exchange (4 key groups x 16 columns x 16 bytes), the
// rescale factors of the 16 columns, and, at a piece end, a 16 x 36-float
// transpose buffer over the same bytes.
constexpr int kValuXchgBytes = 16 * 36 * 4;
constexpr int kValuAlphaOffset = 1024;

__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c, false);
}

template <int D>
struct ValuState {
  static constexpr int CH = D / 16;
  float acc[4][CH];  // lane (c, grp): column 4 grp + j, dim 16 blk + c
  float m;           // running max of the lane's column (log2 units), same in its four lanes
  float l;           // running sum of P over the lane's keys
};

template <int D>
__device__ __forceinline__ void reset_state(ValuState<D>& vs) {
  vs.m = kNegBig;
  vs.l = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int blk = 0; blk < D / 16; ++blk) vs.acc[j][blk] = 0.f;
}

// Lane offsets of the vector-ALU reads within a page tile.  The row key is
// XOR-linear, so key(4 a + b) = key(4 a) ^ key(b) for b < 4; with it, one
// offset per chunk position serves every key and block, and the rest of each
// address is a compile-time immediate.
//   k[w]: row 4 grp + i, chunk u sits at k[u ^ key(i)] + 16 chunks i;
//   v[c]: the transposing read of key group kg, block blk sits at
//         v[2 blk ^ key(4 kg)] + 16 chunks 4 kg (lane 4 e + q of a 16-lane
//         group addresses row 4 kg + e, chunk 2 blk + q / 2, half q % 2).
template <int D>
struct ValuOffsets {
  static constexpr int chunks = D / 8;
  uint32_t k[chunks];
  uint32_t v[chunks];
};

template <int D>
__device__ __forceinline__ void valu_offsets(ValuOffsets<D>& o, int lane) {
  constexpr int chunks = D / 8;
  const int grp = lane >> 4, s = lane & 15, e = s >> 2, q = s & 3;
  const int kgrp = row_key<chunks>(4 * grp);
  const int lv = (q >> 1) ^ row_key<chunks>(e);
#pragma unroll
  for (int w = 0; w < chunks; ++w) {
    o.k[w] = uint32_t(16 * (4 * grp * chunks + (w ^ kgrp)));
    o.v[w] = uint32_t(16 * (e * chunks + (w ^ lv)) + 8 * (q & 1));
  }
}

// O += P V for one step on the vector ALU: lane (c, grp) adds, for columns
// 4 grp + j and dims 16 blk + c, the products over all 32 keys.  px: the
// packed P of every (key group, column).  T: the step ends inside its keys,
// whose V slots past kend may hold anything (0 * NaN is NaN) and are zeroed;
// a separate instance, so the common path reads one key group's V^T at a
// time instead of the whole step's before a branch.
template <int D, bool T>
__device__ __forceinline__ void valu_pv(ValuState<D>& vs, const unsigned char* stage, const ValuOffsets<D>& off,
                                        const u32x4* px, int k0, int kend, int grp) {
  using TG = TileGeom<D>;
  constexpr int CH = D / 16;
  constexpr int chunks = TG::chunks;
  const unsigned char* v0 = stage + 2 * TG::page_bytes;
  const unsigned char* v1 = stage + 3 * TG::page_bytes;
#pragma unroll
  for (int kg = 0; kg < 4; ++kg) {
    u32x4 pj[4];  // P of columns 4 grp + j for key group kg
#pragma unroll
    for (int j = 0; j < 4; ++j) pj[j] = px[16 * kg + 4 * grp + j];
    uint32_t keep[4] = {~0u, ~0u, ~0u, ~0u};
    if constexpr (T) {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2) {
          const int key = k0 + 16 * t + 4 * kg + 2 * h2;  // the word's two keys: key, key + 1
          keep[2 * t + h2] = (key < kend ? 0x0000FFFFu : 0u) | (key + 1 < kend ? 0xFFFF0000u : 0u);
        }
    }
    const int kk = row_key<chunks>(4 * kg);
#pragma unroll
    for (int blk = 0; blk < CH; ++blk) {
      const uint32_t o = off.v[(2 * blk) ^ kk] + 16 * chunks * 4 * kg;
      const s16x4 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4)(v0 + o));
      const s16x4 y = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4)(v1 + o));
      u32x4 vw = __builtin_bit_cast(u32x4, __builtin_shufflevector(x, y, 0, 1, 2, 3, 4, 5, 6, 7));
      if constexpr (T) {
#pragma unroll
        for (int w = 0; w < 4; ++w) vw[w] &= keep[w];
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float acc = vs.acc[j][blk];
#pragma unroll
        for (int w = 0; w < 4; ++w) acc = dot2_bf16(vw[w], pj[j][w], acc);
        vs.acc[j][blk] = acc;
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// One 32-key step of a decode piece on the vector ALU (16 query columns per
// wave, as attend_step with one block).  qrow: the lane's column's Q (D / 8
// chunks); xchg: the wave's LDS exchange area.
template <int D>
__device__ __forceinline__ void attend_step_valu(ValuState<D>& vs, const unsigned char* stage,
                                                 const u32x4 (&qrow)[D / 8], const ValuOffsets<D>& off, int lim,
                                                 int k0, int kend, bool causal, int lane, float scale_log2,
                                                 unsigned char* xchg) {
  using TG = TileGeom<D>;
  constexpr int CH = D / 16;
  constexpr int chunks = TG::chunks;
  const int col = lane & 15, grp = lane >> 4;
  const bool tail = k0 + kStepKeys > kend;
  float v[8];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const unsigned char* krow = stage + t * TG::page_bytes + 16 * chunks * i;
      const int ki = row_key<chunks>(i);
      float sc = 0.f;
#pragma unroll
      for (int u = 0; u < chunks; ++u) {
        const u32x4 kw = *reinterpret_cast<const u32x4*>(krow + off.k[u ^ ki]);
#pragma unroll
        for (int w = 0; w < 4; ++w) sc = dot2_bf16(kw[w], qrow[u][w], sc);
      }
      v[4 * t + i] = sc;
    }
  if (tail || causal) {
    PFX_KEEP_BRANCH();
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = k0 + 16 * t + 4 * grp + i;
        if (key >= kend || (causal && key > lim)) v[4 * t + i] = -INFINITY;
      }
  }
  float mx = v[0];
#pragma unroll
  for (int i = 1; i < 8; ++i) mx = __builtin_elementwise_maximum(mx, v[i]);
  if (__any(mx * scale_log2 > vs.m + kRescaleSlack)) {
    PFX_KEEP_BRANCH();
    mx = column_max(mx) * scale_log2;
    const bool raise = mx > vs.m + kRescaleSlack;
    const float mnew = raise ? mx : vs.m;
    const float alpha = fast_exp2(vs.m - mnew);
    vs.l *= alpha;
    vs.m = mnew;
    // The lane's accumulators belong to columns 4 grp .. 4 grp + 3.
    float* al = reinterpret_cast<float*>(xchg + kValuAlphaOffset);
    if (grp == 0) al[col] = alpha;
    wave_lds_sync();
    const f32x4 a4 = reinterpret_cast<const f32x4*>(al)[grp];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int blk = 0; blk < CH; ++blk) vs.acc[j][blk] *= a4[j];
    wave_lds_sync();
  }
  const float neg_m = -vs.m;
  float pr[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) pr[j] = fast_exp2(fmaf(v[j], scale_log2, neg_m));
  const u32x4 pw = {pack_bf16(pr[0], pr[1]), pack_bf16(pr[2], pr[3]), pack_bf16(pr[4], pr[5]), pack_bf16(pr[6], pr[7])};
  // The row sum of the rounded P, as the products see it.
  float ps = 0.f;
#pragma unroll
  for (int w = 0; w < 4; ++w)
    ps += __builtin_bit_cast(float, pw[w] << 16) + __builtin_bit_cast(float, pw[w] & 0xFFFF0000u);
  vs.l += ps;
  u32x4* px = reinterpret_cast<u32x4*>(xchg);  // [key group][column]
  px[16 * grp + col] = pw;
  wave_lds_sync();
  if (tail) {
    PFX_KEEP_BRANCH();
    valu_pv<D, true>(vs, stage, off, px, k0, kend, grp);
  } else {
    valu_pv<D, false>(vs, stage, off, px, k0, kend, grp);
  }
  wave_lds_sync();
}

// End of a piece on the vector ALU: the column sum l, and the accumulators
// transposed into the MFMA state layout (o[blk][i] = dim 16 blk + 4 grp + i
// of column col), 32 dims at a time through a [16 columns][36 floats]
// buffer (the padding spreads the 64 lanes' stores over all banks).
template <int D>
__device__ __forceinline__ void valu_finish(const ValuState<D>& vs, unsigned char* xchg, int lane, f32x4 (&o)[D / 16],
                                            float& l) {
  constexpr int CH = D / 16;
  const int col = lane & 15, grp = lane >> 4;
  l = column_sum(vs.l);
  float* tb = reinterpret_cast<float*>(xchg);
#pragma unroll
  for (int p = 0; p < CH / 2; ++p) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int bb = 0; bb < 2; ++bb) tb[(4 * grp + j) * 36 + 16 * bb + col] = vs.acc[j][2 * p + bb];
    wave_lds_sync();
#pragma unroll
    for (int bb = 0; bb < 2; ++bb) o[2 * p + bb] = *reinterpret_cast<const f32x4*>(tb + col * 36 + 16 * bb + 4 * grp);
    wave_lds_sync();
  }
}

// Two consecutive 32-key steps of an extend block under one barrier,
// against the wave's QB blocks of 16 query columns (blocks past the wave's
// columns compute on zero queries and are never written):
//   S^T = K Q^T: lane (col, grp) gets the scores of keys 16 t + 4 grp + i;
//   online softmax in log2 units, the maximum raised lazily: one maximum
//   over the 64 keys, and the cross-lane column maximum taken only when some
//   lane passes m + slack;
//   O^T += V^T P^T with P from the lane's own scores and V^T read by
//   ds_read_b64_tr_b16 (accumulator [blk][i] = dim 16 blk + 4 grp + i), and
//   the row sums of P on the matrix unit (an A operand whose row 0 is ones).
// The rare paths (masking on diagonal and tail steps, raising the maximum,
// zeroing V past the end) are one branch each.  V^T of the second step is
// read after the first step's products, so the two operand sets share
// registers.
template <int D, int QB>
__device__ __forceinline__ void extend_pair(WaveState<D, QB>& ws, const unsigned char* st0,
                                            const unsigned char* st1, const bf16x8 (&qf)[QB][D / 32],
                                            const int (&lim)[QB], const Item& it, int st, bool two,
                                            const StepMarks& mk, int lane, float scale_log2) {
  using TG = TileGeom<D>;
  constexpr int KS = D / 32;
  constexpr int CH = D / 16;
  const int col = lane & 15, grp = lane >> 4;
  f32x4 sc[2][QB][2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const unsigned char* stage = u ? st1 : st0;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      u32x4 kf[KS];
#pragma unroll
      for (int s = 0; s < KS; ++s)
        kf[s] = *reinterpret_cast<const u32x4*>(stage + t * TG::page_bytes +
                                                16 * swizzled_slot<TG::chunks>(col, 4 * s + grp));
#pragma unroll
      for (int b = 0; b < QB; ++b) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KS; ++s)
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kf[s]), qf[b][s], acc, 0, 0, 0);
        sc[u][b][t] = acc;
      }
    }
  }
  // An odd last step pairs with an empty one (no visible key: all its scores
  // -inf, its V zeroed).
  if (!two || st + 1 >= mk.diag || st == mk.tail0 || st + 1 == mk.tail0 || st == mk.tail1 || st + 1 == mk.tail1) {
    PFX_KEEP_BRANCH();
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      StepPos p = step_pos(it, st, mk.s0_steps);
      if (u) p = two ? step_pos(it, st + 1, mk.s0_steps) : StepPos{p.list_off, p.kend, p.kend, p.seg};
#pragma unroll
      for (int b = 0; b < QB; ++b) {
        const int lim_b = p.seg == 1 ? lim[b] : 0x7fffffff;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int key = p.k0 + 16 * t + 4 * grp + i;
            if (key >= p.kend || key > lim_b) sc[u][b][t][i] = -INFINITY;
          }
      }
    }
  }
  float mx[QB];
  bool pass = false;
#pragma unroll
  for (int b = 0; b < QB; ++b) {
    // IEEE maximum (NaN-propagating, gfx950 v_maximum3_f32): fmaxf would put a
    // NaN canonicalisation in front of every MFMA result it reads.
    float x[16];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) x[8 * u + 4 * t + i] = sc[u][b][t][i];
#pragma unroll
    for (int w = 8; w >= 1; w /= 2)
#pragma unroll
      for (int i = 0; i < w; ++i) x[i] = __builtin_elementwise_maximum(x[i], x[i + w]);
    mx[b] = x[0];
    pass = pass || mx[b] * scale_log2 > ws.m[b] + kRescaleSlack;  // scale > 0
  }
  if (__any(pass)) {
    PFX_KEEP_BRANCH();
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      const float cm = column_max(mx[b]) * scale_log2;
      const float mnew = cm > ws.m[b] + kRescaleSlack ? cm : ws.m[b];
      const float alpha = fast_exp2(ws.m[b] - mnew);  // 1 for columns that keep their maximum
      ws.lv[b][0] *= alpha;                           // rows other than 0 stay zero
#pragma unroll
      for (int blk = 0; blk < CH; ++blk) ws.acc[b][blk] *= alpha;
      ws.m[b] = mnew;
    }
  }
  const uint32_t one2 = col == 0 ? 0x3F803F80u : 0u;  // bf16 1.0 pairs in row 0
  const bf16x8 ones_row0 = __builtin_bit_cast(bf16x8, u32x4{one2, one2, one2, one2});
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const unsigned char* stage = u ? st1 : st0;
    if (u) asm volatile("" ::: "memory");  // the second step's V reads stay after the first step's products
    bf16x8 vop[CH];
#pragma unroll
    for (int blk = 0; blk < CH; ++blk)
      vop[blk] = v_operand_tr<D>(stage + 2 * TG::page_bytes, stage + 3 * TG::page_bytes, blk, lane);
    if ((u == 1 && !two) || st + u == mk.tail0 || st + u == mk.tail1) {
      PFX_KEEP_BRANCH();
      const StepPos p = u == 1 && !two ? StepPos{0, 0, 0, 0} : step_pos(it, st + u, mk.s0_steps);
      zero_v_tail<D>(vop, p.k0, p.kend, grp);
    }
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      const float neg_m = -ws.m[b];
      float pr[8];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) pr[4 * t + i] = fast_exp2(fmaf(sc[u][b][t][i], scale_log2, neg_m));
      const u32x4 pw = {pack_bf16(pr[0], pr[1]), pack_bf16(pr[2], pr[3]), pack_bf16(pr[4], pr[5]),
                        pack_bf16(pr[6], pr[7])};
      const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
#pragma unroll
      for (int blk = 0; blk < CH; ++blk)
        ws.acc[b][blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop[blk], pb, ws.acc[b][blk], 0, 0, 0);
      ws.lv[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones_row0, pb, ws.lv[b], 0, 0, 0);
    }
  }
}

// Normalise a wave's block and write it as final rows (bf16 o, lse): lane
// (col, grp) holds dims 16 blk + 4 grp + i of its column, four consecutive
// dims per block.  The column's output row is orow; invalid columns
// (padding) write nothing.
template <int D>
__device__ __forceinline__ void write_rows(const AttnArgs& a, const f32x4 (&acc)[D / 16], float m, float l_lane,
                                           int orow, bool valid, int grp) {
  constexpr int CH = D / 16;
  const float l = column_sum(l_lane);
  if (!valid) return;
  const float inv = l > 0.f ? 1.0f / l : 0.f;
  const float lse_nat = l > 0.f ? (m + log2f(l)) * kLn2 : -INFINITY;
  uint16_t* out = a.o + size_t(orow) * D + 4 * grp;
#pragma unroll
  for (int blk = 0; blk < CH; ++blk) {
    u32x2 w = {pack_bf16(acc[blk][0] * inv, acc[blk][1] * inv), pack_bf16(acc[blk][2] * inv, acc[blk][3] * inv)};
    *reinterpret_cast<u32x2*>(out + 16 * blk) = w;
  }
  if (a.lse && grp == 0) a.lse[orow] = lse_nat;
}

// The page ids of an extend block -- its page table, segment 0's pages then
// segment 1's -- reach each wave as it needs them: a window of 64
// consecutive entries, one per lane (`cur`, entries w0 .. w0 + 63), and the
// window after it (`next`), requested when the wave moves into `cur`, about
// 32 steps before it is needed.  So a block may stream any number of pages.
struct PageWindow {
  const int32_t* list;  // the plan's page list
  int32_t s0_at, s1_at; // where the table's entries of segment 0 and of segment 1 start in it
  int32_t p0n, ntab;    // entries of segment 0; of the whole table
  int32_t w0;           // first entry held in cur
  int32_t cur, next;
};

__device__ __forceinline__ int window_entry(const PageWindow& w, int e) {
  if (e >= w.ntab) return 0;
  return e < w.p0n ? w.list[w.s0_at + e] : w.list[w.s1_at + e - w.p0n];
}

// Page-table entry of this wave's tile (wave & 1) of step st.
__device__ __forceinline__ int step_entry(const StepMarks& mk, int st, int wave) {
  const int t = wave & 1;
  int idx = 2 * st + t + (st >= mk.s0_steps ? mk.d1 : 0);
  if (t == 1 && (st == mk.half0 || st == mk.half1)) idx -= 1;  // a missing second page re-reads the first (masked later)
  return idx;
}

// Issue this wave's share of an extend block's step st into a stage buffer:
// tile (wave & 1) of K (waves 0, 1) or of V (waves 2, 3), from page `page`.
template <int D>
__device__ __forceinline__ void issue_block_copy(unsigned char* stage, const AttnArgs& a, int page, int h, int wave,
                                                 const uint32_t (&voff)[TileGeom<D>::loads_per_wave]) {
  using TG = TileGeom<D>;
  const uint16_t* base = ((wave >> 1) ? a.vpool : a.kpool) + (size_t(page) * a.hkv + h) * (16 * D);
  copy_block_to_lds(base, voff, lds_address(stage) + wave * TG::page_bytes);
}

// Step st's page through the window.  Entries grow by at most 3 from one of
// this wave's steps to the next, so a step either finds its entry in cur or
// moves one window on (its successor, requested 64 entries earlier, has
// arrived: every pair waits for all of the wave's memory operations).
__device__ __forceinline__ int window_page(PageWindow& pw, int idx, int lane) {
  if (idx >= pw.w0 + 64) {
    pw.w0 += 64;
    pw.cur = pw.next;
    pw.next = window_entry(pw, pw.w0 + 64 + lane);
  }
  return __builtin_amdgcn_readfirstlane(__builtin_amdgcn_readlane(pw.cur, idx - pw.w0));
}

// LDS bytes of an extend block: the ring.
template <int D>
constexpr int extend_smem_bytes() { return kStages * TileGeom<D>::stage_bytes; }

// One extend block (QBW blocks of 16 columns per wave): its K/V streams once
// through the LDS ring, two steps at a time; at every pair each wave waits
// for its own copies, all waves meet (the pair's stages complete everywhere,
// the previous pair's stages consumed), those are refilled two steps ahead,
// and every wave multiplies the pair against its own columns.
template <int D, int QBW>
__device__ __forceinline__ void extend_block(const AttnArgs& a, const Item* itp, unsigned char* smem) {
  using TG = TileGeom<D>;
  constexpr int KS = D / 32;
  constexpr int NS = kStages;
  auto ring = reinterpret_cast<unsigned char (*)[TG::stage_bytes]>(smem);
  const int lead = itp->first_pages[threadIdx.x & (kItemPages - 1)];  // issued before the block's scalar load
  const Item it = *itp;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int h = it.kv_head;
  const int G = a.group;

  // The block's page table: segment 0's pages, then segment 1's, read
  // through a window of 64 entries per wave (the first two windows now).
  const int p0b = it.s0_kbeg >> 4;
  const int p0n = it.s0_kend > it.s0_kbeg ? ((it.s0_kend + 15) >> 4) - p0b : 0;
  const int p1b = it.s1_kbeg >> 4;
  const int p1n = it.s1_kend > it.s1_kbeg ? ((it.s1_kend + 15) >> 4) - p1b : 0;
  PageWindow pw;
  pw.list = a.plan.page_list;
  pw.s0_at = it.s0_page_off + p0b;
  pw.s1_at = it.s1_page_off + p1b;
  pw.p0n = p0n;
  pw.ntab = p0n + p1n;
  pw.w0 = 0;
  pw.cur = window_entry(pw, lane);
  pw.next = window_entry(pw, 64 + lane);

  // This wave's query columns: blocks wave*QBW .. wave*QBW + QBW - 1.
  const int ncols = it.row_count * G;
  int nb = (ncols - wave * QBW * kTileCols + kTileCols - 1) / kTileCols;
  nb = nb < 0 ? 0 : (nb > QBW ? QBW : nb);
  bf16x8 qf[QBW][KS];
  int lim[QBW];
  int orow[QBW];
  int prow[QBW];  // wide prefix blocks: the partial row of each column
#pragma unroll
  for (int b = 0; b < QBW; ++b) {
    const int c = (wave * QBW + b) * kTileCols + col;
    int j = c >> a.group_shift;
    const int gg = c & (G - 1);
    if (j >= it.row_count) j = 0;
    const int tok = it.tok0 >= 0 ? it.tok0 + j : a.plan.row_tok[it.row_begin + j];
    prow[b] = it.out_slot >= 0 ? a.plan.row_out[it.row_begin + j] + gg : -1;
    lim[b] = tok + it.causal_base;
    orow[b] = tok * a.hq + h * G + gg;
    if (b < nb) {
      const uint16_t* qp = a.q + size_t(orow[b]) * D + 8 * grp;
#pragma unroll
      for (int s = 0; s < KS; ++s) qf[b][s] = *reinterpret_cast<const bf16x8*>(qp + 32 * s);
    } else {
#pragma unroll
      for (int s = 0; s < KS; ++s) qf[b][s] = bf16x8{};
    }
  }
  // Block 0, column 0 holds the wave's lowest token (padding columns repeat
  // the item's first row).
  const int lim_lo = __builtin_amdgcn_readfirstlane(lim[0]);
  WaveState<D, QBW> ws;
  reset_state(ws);
  const StepMarks mk = step_marks(it, p0n, lim_lo);
  const int nsteps = mk.nsteps;
  uint32_t voff[TG::loads_per_wave];
  block_lane_offsets<D>(voff, lane);
  // The first two steps' pages are among the leading ids (they travel in
  // the block record, one per lane): request them before the page windows
  // arrive.
  for (int st = 0; st < 2 && st < nsteps; ++st)
    issue_block_copy<D>(ring[st], a, __builtin_amdgcn_readfirstlane(__builtin_amdgcn_readlane(lead, step_entry(mk, st, wave))),
                        h, wave, voff);
  // Two steps per barrier: at pair q (steps 2q, 2q + 1) wait for both
  // stages, meet (so the stages of the previous pair are free), refill them
  // with steps 2q + 2 and 2q + 3, and run the pair.  Unrolled by two pairs,
  // so every copy of the body works on fixed stages and its LDS addresses
  // are a lane offset plus an immediate.
  static_assert(NS == 4, "pairs of steps in a ring of four stages");
  for (int st0 = 0; st0 < nsteps; st0 += 4) {
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int st = st0 + 2 * k;
      if (st >= nsteps) break;
      const bool two = st + 1 < nsteps;
      wait_vmcnt(0);
      __syncthreads();
      if (st + 2 < nsteps)
        issue_block_copy<D>(ring[(2 * k + 2) % NS], a, window_page(pw, step_entry(mk, st + 2, wave), lane), h, wave,
                            voff);
      if (st + 3 < nsteps)
        issue_block_copy<D>(ring[(2 * k + 3) % NS], a, window_page(pw, step_entry(mk, st + 3, wave), lane), h, wave,
                            voff);
      // An odd last step pairs with an empty one (its stage is not being
      // refilled).
      if (nb > 0) extend_pair<D, QBW>(ws, ring[2 * k], ring[2 * k + 1], qf, lim, it, st, two, mk, lane, a.scale_log2);
    }
  }
#pragma unroll
  for (int b = 0; b < QBW; ++b) {
    const int c = (wave * QBW + b) * kTileCols + col;
    const bool valid = b < nb && (c >> a.group_shift) < it.row_count;
    if (it.out_slot < 0) {
      write_rows<D>(a, ws.acc[b], ws.m[b], ws.lv[b][0], orow[b], valid, grp);
    } else if (valid) {
      // A wide prefix block's state, as a decode piece leaves it:
      // the accumulators divided by l as bf16 units of the partial layout,
      // (m, l) once per column.
      const float l = column_sum(ws.lv[b][0]);  // the column sum sits in the group-0 lanes
      store_partial<D>(a.plan.o_part, size_t(prow[b]), c & (G - 1), G, grp, ws.acc[b], l > 0.f ? 1.0f / l : 0.f);
      if (grp == 0) *reinterpret_cast<f32x2*>(a.plan.l_part + 2 * size_t(prow[b])) = f32x2{ws.m[b], l};
    }
  }
}

// Extend blocks: final rows, 32 query columns per wave.
template <int D>
__global__ __launch_bounds__(256, 2) void extend_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(1024))) unsigned char smem[extend_smem_bytes<D>()];
  extend_block<D, 2>(a, a.plan.items + blockIdx.x, smem);
}

// ---------------------------------------------------------------------------
// Decode.
//
// S workgroups (by default one per piece), each running a fixed list of
// pieces through one LDS ring.  Round r of the longest-first list gives
// workgroup b piece r S + b on even rounds and r S + S - 1 - b on odd ones.
// Every piece contributes a Q stage (its query rows, each wave's 16
// columns in its quarter of the stage) and then its K/V steps, and stage u
// is refilled with stage u + kDecodeStages - 1 whatever piece that belongs to, so
// a piece boundary does not drain the ring.  A piece's descriptor (header, rows, page blocks)
// comes into one of kPieceSlots LDS slots by a direct copy that wave 0
// issues with the Q stage two pieces earlier; it is complete once that stage
// has been waited for, long before the issue reaches the piece.
// ---------------------------------------------------------------------------
// The decode ring has three stages (two in flight while one is consumed):
// a decode step is short, and a fourth stage measured 1-2% slower (decode
// steps queued behind the others' requests rather than adding bandwidth).
constexpr int kDecodeStages = 3;

// V: the decode pieces run on the vector ALU, with a per-wave exchange area.
template <int D, bool V>
constexpr int decode_smem_bytes() {
  return kDecodeStages * TileGeom<D>::stage_bytes + kPieceSlots * int(sizeof(Seg)) + (V ? 4 * kValuXchgBytes : 0);
}

// Piece of workgroup b at position n of its list (>= num_pieces: none).
__device__ __forceinline__ int piece_of(int b, int n, int S) { return n * S + ((n & 1) ? S - 1 - b : b); }

// Block ids of this wave's tile (wave & 1) for the steps of a piece, one per
// lane: a step finds its page with v_readlane.
__device__ __forceinline__ int piece_window(const Seg& sg, int wave, int lane) {
  return lane < kPieceSteps ? sg.steps[2 * lane + (wave & 1)] : 0;
}

// Where a suffix piece's new tokens are, for the folded-in append: keys
// [first_new, kend) of its item (the item's last ncols / G keys); first_new
// is past every key for other pieces.
struct NewRows {
  int32_t k0, kend, first_new, head;
};

// Issue this wave's copies of stage k of a piece (k < 0: its Q stage);
// returns how many copies it issued (a wave with no columns copies no Q).
// F: the append is folded in, and a tile holding new tokens takes their
// rows from k_new / v_new.
template <int D, bool F>
__device__ __forceinline__ int issue_piece_stage(unsigned char* stage, const AttnArgs& a, const Seg& sg, int win,
                                                 int k, int ncols, int qh0, int wave, int lane,
                                                 const uint32_t (&voff)[TileGeom<D>::loads_per_wave],
                                                 const NewRows& nr) {
  using TG = TileGeom<D>;
  const uint32_t dst = lds_address(stage) + wave * TG::page_bytes;
  if (k >= 0) {
    // K/V: tile (wave & 1) of K (waves 0, 1) or V (waves 2, 3), swizzled.
    const int blk = __builtin_amdgcn_readlane(win, k);
    const uint16_t* base = ((wave >> 1) ? a.vpool : a.kpool) + size_t(blk) * (16 * D);
    if constexpr (F) {
      const int tk0 = nr.k0 + kStepKeys * k + 16 * (wave & 1);
      if (tk0 + 16 > nr.first_new && tk0 < nr.kend) {
        // This tile holds some of the piece's new tokens: their rows come
        // from k_new / v_new, the others from the pool, one copy per lane
        // with its own address.
        PFX_KEEP_BRANCH();
        const uint16_t* fresh = (wave >> 1) ? a.v_new : a.k_new;
#pragma unroll
        for (int j = 0; j < TG::loads_per_wave; ++j) {
          const int t = (64 * j + lane) / TG::chunks;
          const int c = (lane % TG::chunks) ^ row_key<TG::chunks>(t);
          const int key = tk0 + t;
          const bool is_new = key >= nr.first_new && key < nr.kend;
          const int row = is_new ? key - nr.first_new : 0;
          const uint16_t* src =
              is_new ? fresh + (size_t(sg.tok[row]) * a.hkv + nr.head) * D + 8 * c : base + t * D + 8 * c;
          copy16_to_lds(src, dst + 1024 * j);
        }
        return TG::loads_per_wave;
      }
    }
    copy_block_to_lds(base, voff, dst);
    return TG::loads_per_wave;
  }
  // Q: chunk (p % chunks) of this wave's column p / chunks at 16 p; padding
  // columns repeat the piece's first column.
  if (16 * wave >= ncols) return 0;
#pragma unroll
  for (int j = 0; j < TG::loads_per_wave; ++j) {
    const int q = 64 * j + lane;
    int cl = 16 * wave + q / TG::chunks;
    cl = cl < ncols ? cl : 0;
    const uint16_t* src =
        a.q + (size_t(sg.tok[cl >> a.group_shift]) * a.hq + qh0 + (cl & (a.group - 1))) * D + 8 * (q % TG::chunks);
    copy16_to_lds(src, dst + 1024 * j);
  }
  return TG::loads_per_wave;
}

// F: the append is folded in.  W: the launch starts with wide prefix blocks.
// V: the pieces run on the vector ALU (no wide blocks then).
template <int D, bool F, bool W, bool V>
__global__ __launch_bounds__(256, 2) void decode_kernel(AttnArgs a) {
  static_assert(!(V && W), "wide blocks run on the matrix unit");
  using TG = TileGeom<D>;
  constexpr int KS = D / 32;
  constexpr int CH = D / 16;
  constexpr int NS = kDecodeStages;
  constexpr int K = kPieceSlots;
  constexpr int kVecs = int(sizeof(Seg)) / 16;
  static_assert(kVecs > 64 && kVecs <= 128, "a descriptor is two copy instructions");
  // Wide prefix blocks run the extend block's four-stage ring in the same bytes.
  constexpr int kSmem = W ? std::max(extend_smem_bytes<D>(), decode_smem_bytes<D, V>()) : decode_smem_bytes<D, V>();
  __shared__ __attribute__((aligned(1024))) unsigned char smem[kSmem];
  if constexpr (W) {
    if (int(blockIdx.x) < a.num_wide) {
      // A wide prefix block: 128 decode columns against one piece of their
      // agent's prefix, the extend block's two-steps-per-barrier pipeline.
      extend_block<D, 2>(a, a.plan.items + a.wide_first + blockIdx.x, smem);
      return;
    }
  }
  auto ring = reinterpret_cast<unsigned char (*)[TG::stage_bytes]>(smem);
  Seg* slots = reinterpret_cast<Seg*>(smem + NS * TG::stage_bytes);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int S = int(gridDim.x) - a.num_wide, b = int(blockIdx.x) - a.num_wide;
  const int np = a.num_pieces;

  // The first two descriptors.
  for (int i = threadIdx.x; i < 2 * kVecs; i += 256) {
    const int piece = piece_of(b, i / kVecs, S);
    if (piece < np)
      reinterpret_cast<u32x4*>(&slots[i / kVecs])[i % kVecs] =
          reinterpret_cast<const u32x4*>(&a.plan.segs[piece])[i % kVecs];
  }
  __syncthreads();

  uint32_t voff[TG::loads_per_wave];
  block_lane_offsets<D>(voff, lane);
  // Issue side: piece iord of the list, its next stage ik (-1: Q), and what
  // the issue needs of it.
  int iord = 0, ik = -1, inst = 0, incols = 0, iqh0 = 0, iwin = 0;
  NewRows inew = {0, 0, 0x7fffffff, 0};
  bool in_piece = false, ended = false;
  // Per ring stage (16 bits each), what was issued into it: bit 9 valid,
  // bits 7-8 slot, bits 0-6 step + 1 (0: Q).  ops: copies this wave issued
  // per issue opportunity, 8 bits each, newest lowest.
  uint64_t ent = 0;
  uint32_t ops = 0;
  int pending = 0;

  auto issue_next = [&](int r) {
    uint32_t code = 0;
    int n_ops = 0;
    if (!in_piece && !ended) {
      if (piece_of(b, iord, S) >= np) {
        ended = true;
      } else {
        const Seg& sg = slots[iord % K];
        const i32x4 h = *reinterpret_cast<const i32x4*>(&sg.h);  // kind, kv_head, ncols, nsteps
        iqh0 = __builtin_amdgcn_readfirstlane(h[1]) * a.group;
        incols = __builtin_amdgcn_readfirstlane(h[2]);
        inst = __builtin_amdgcn_readfirstlane(h[3]);
        iwin = piece_window(sg, wave, lane);
        if constexpr (F) {
          const i32x4 h1 = *reinterpret_cast<const i32x4*>(&sg.h.k0);  // k0, kend, causal_base, slot
          inew.k0 = __builtin_amdgcn_readfirstlane(h1[0]);
          inew.kend = __builtin_amdgcn_readfirstlane(h1[1]);
          inew.first_new = __builtin_amdgcn_readfirstlane(h[0]) == kSuffixItem ? inew.kend - (incols >> a.group_shift)
                                                                             : 0x7fffffff;
          inew.head = __builtin_amdgcn_readfirstlane(h[1]);
        }
        ik = -1;
        in_piece = true;
      }
    }
    if (in_piece) {
      const int q = iord % K;
      n_ops = issue_piece_stage<D, F>(ring[r], a, slots[q], iwin, ik, incols, iqh0, wave, lane, voff, inew);
      if (ik < 0 && wave == 0) {
        // The descriptor two pieces ahead, into the slot of the piece two back.
        const int nxt = piece_of(b, iord + 2, S);
        if (nxt < np) {
          // Two copies: 16-byte chunks lane and 64 + lane (lanes 0 .. kVecs - 65).
          const unsigned char* src = reinterpret_cast<const unsigned char*>(&a.plan.segs[nxt]);
          const uint32_t dst = lds_address(reinterpret_cast<const unsigned char*>(&slots[(iord + 2) % K]));
          copy16_to_lds(src + 16 * lane, dst);
          if (lane < kVecs - 64) copy16_to_lds(src + 16 * (64 + lane), dst + 1024);
          n_ops += 2;
        }
      }
      code = 0x200u | (uint32_t(q) << 7) | uint32_t(ik + 1);
      ++pending;
      if (++ik == inst) {
        ++iord;
        in_piece = false;
      }
    }
    ent = (ent & ~(uint64_t(0xFFFFu) << (16 * r))) | (uint64_t(code) << (16 * r));
    ops = (ops << 8) | uint32_t(n_ops);
  };
  for (int u = 0; u < NS - 1; ++u) issue_next(u);

  std::conditional_t<V, ValuState<D>, WaveState<D, 1>> ws;
  reset_state(ws);
  unsigned char* xchg = smem + NS * TG::stage_bytes + K * int(sizeof(Seg)) + wave * kValuXchgBytes;
  bf16x8 qf[1][KS];
  u32x4 qrow[TG::chunks];  // vector-ALU engine: the lane's whole Q row
  ValuOffsets<D> voffs;
  if constexpr (V) valu_offsets<D>(voffs, lane);
  int lim[1] = {0};
  int orow = 0, k0 = 0, kend = 0, causal = 0, cnst = 0;
  bool has_cols = false, valid = false;
  // Unrolled over the ring, so that every stage's LDS addresses are a lane
  // offset plus an immediate.
  while (!(ended && pending == 0)) {
#pragma unroll
    for (int r = 0; r < NS; ++r) {
      if (ended && pending == 0) break;
      // Stage in ring slot r: only the copies of the issue opportunities after it (the
      // newest NS - 2 entries of ops) may still be pending.
      int later = 0;
#pragma unroll
      for (int i = 0; i < NS - 2; ++i) later += (ops >> (8 * i)) & 0xFFu;
      wait_vmcnt(later);
      __syncthreads();
      issue_next((r + NS - 1) % NS);

      const uint32_t code = uint32_t(ent >> (16 * r)) & 0xFFFFu;
      const unsigned char* stage = ring[r];
      if (code & 0x200u) {
        --pending;
        const Seg& sg = slots[(code >> 7) & 3u];
        const int k = int(code & 127u) - 1;
        if (k < 0) {
          // A piece starts: its columns, limits, output rows and Q.
          const i32x4 h0 = *reinterpret_cast<const i32x4*>(&sg.h);       // kind, kv_head, ncols, nsteps
          const i32x4 h1 = *reinterpret_cast<const i32x4*>(&sg.h.k0);    // k0, kend, causal_base, slot
          const i32x4 h2 = *reinterpret_cast<const i32x4*>(&sg.h.item);  // item, piece, causal, -
          const int ncols = __builtin_amdgcn_readfirstlane(h0[2]);
          cnst = __builtin_amdgcn_readfirstlane(h0[3]);
          k0 = __builtin_amdgcn_readfirstlane(h1[0]);
          kend = __builtin_amdgcn_readfirstlane(h1[1]);
          causal = __builtin_amdgcn_readfirstlane(h2[2]);
          // New tokens of a suffix piece: its item's last ncols / G keys.
          has_cols = 16 * wave < ncols;
          const int c = 16 * wave + col;
          valid = c < ncols;
          const int j = valid ? c >> a.group_shift : 0;
          const int tok = sg.tok[j];
          lim[0] = causal ? tok + __builtin_amdgcn_readfirstlane(h1[2]) : 0x7fffffff;
          orow = sg.out[j] + (c & (a.group - 1));
          if (has_cols) {
            const unsigned char* qb = stage + wave * TG::page_bytes;
            if constexpr (V) {
#pragma unroll
              for (int u = 0; u < TG::chunks; ++u)
                qrow[u] = *reinterpret_cast<const u32x4*>(qb + 16 * (col * TG::chunks + u));
            } else {
#pragma unroll
              for (int s = 0; s < KS; ++s)
                qf[0][s] = *reinterpret_cast<const bf16x8*>(qb + 16 * (col * TG::chunks + 4 * s + grp));
            }
          }
        } else {
          if (has_cols) {
            if constexpr (V)
              attend_step_valu<D>(ws, stage, qrow, voffs, lim[0], k0 + kStepKeys * k, kend, causal != 0, lane,
                                  a.scale_log2, xchg);
            else
              attend_step<D, 1>(ws, stage, qf, lim, k0 + kStepKeys * k, kend, causal != 0, 1, lane, a.scale_log2);
            if (k == cnst - 1) {
              // The piece's state goes out as it stands: the accumulators
              // divided by l as bf16 units of the partial layout, (m, l) once
              // per column.
              float l, m;
              f32x4 acc[CH];
              if constexpr (V) {
                valu_finish<D>(ws, xchg, lane, acc, l);
                m = ws.m;
              } else {
                l = column_sum(ws.lv[0][0]);  // the column sum sits in the group-0 lanes
                m = ws.m[0];
#pragma unroll
                for (int jj = 0; jj < CH; ++jj) acc[jj] = ws.acc[0][jj];
              }
              if (valid) {
                store_partial<D>(a.plan.o_part, size_t(orow), (16 * wave + col) & (a.group - 1), a.group, grp, acc,
                                 l > 0.f ? 1.0f / l : 0.f);
                if (grp == 0) *reinterpret_cast<f32x2*>(a.plan.l_part + 2 * size_t(orow)) = f32x2{m, l};
              }
              reset_state(ws);
            }
          }
        }
      }
    }
  }
}

// Decode rows: the log-sum-exp merge of the pieces' states (softmax over a
// union of disjoint key ranges, recombined exactly from each range's maximum,
// sum and weighted values; the paper itself states no attention numerics).
// One thread per (token, query head, group grp, block pair): it
// reads elements i = 0..3 of blocks blk, blk + 1 of every piece, i.e. dims
// 16 blk + 4 grp + i and 16 (blk + 1) + 4 grp + i, and writes them as two
// runs of four bf16.  The first kMergeBatch pieces are all requested before
// any is used.
constexpr int kMergeBatch = 8;

// F: the append of this step is folded in.  The decode launch read every
// decode token's new K/V straight from k_new / v_new; the merge, which runs
// after it, writes them into their pool slots (2 Hkv D / 8 chunks of 16
// bytes per token, spread over the token's threads).
template <int D, bool F>
__global__ __launch_bounds__(128) void merge_rows_kernel(AttnArgs a, int n_tok) {
  constexpr int CH = D / 16;
  constexpr int SL = D / 8;  // threads per row: 4 groups x CH/2 pairs
  const size_t t = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= size_t(n_tok) * a.hq * SL) return;
  const int sl = int(t % SL);
  const int grp = sl / (CH / 2), blk = 2 * (sl % (CH / 2));
  const int qh = int((t / SL) % a.hq);
  const int m = int(t / (size_t(SL) * a.hq));
  // The append's chunks (at most two per thread: 2 Hkv <= 2 Hq), loaded
  // beside the merge's own loads and stored at the end.
  constexpr int kAppendPerThread = 2;
  u32x4 app_val[kAppendPerThread];
  uint16_t* app_dst[kAppendPerThread] = {nullptr, nullptr};
  if constexpr (F) {
    const int tok = a.merge_tok_is_row ? m : a.plan.merge_tok[m];
    const int slot = a.plan.tok_slot[tok];
    const int per = a.hkv * SL;  // chunks of K (or V) per token
#pragma unroll
    for (int i = 0; i < kAppendPerThread; ++i) {
      const int e = qh * SL + sl + i * a.hq * SL;
      if (e < 2 * per) {
        const bool is_v = e >= per;
        const int hh = (e % per) / SL, c = e % SL;
        app_val[i] = *reinterpret_cast<const u32x4*>((is_v ? a.v_new : a.k_new) + (size_t(tok) * a.hkv + hh) * D + 8 * c);
        app_dst[i] = const_cast<uint16_t*>(is_v ? a.vpool : a.kpool) +
                     ((size_t(slot >> 4) * a.hkv + hh) * 16 + (slot & 15)) * D + 8 * c;
      }
    }
  }
  const size_t unit = size_t(m) * a.hkv + (qh >> a.group_shift);
  const MergeHead mh = a.merge_parts ? MergeHead{int32_t(unit) * a.merge_parts, a.merge_parts} : a.plan.merge_head[unit];
  const int tok = F && a.merge_tok_is_row ? m : a.plan.merge_tok[m];
  const size_t row0 = size_t(mh.base) * a.group + (qh & (a.group - 1));
  const size_t stride = size_t(a.group);  // rows between slots
  // Unit 4 (blk / 2) + grp of the row in slot 0: blocks blk and blk + 1.
  const uint16_t* op =
      part_unit0(a.plan.o_part, row0, qh & (a.group - 1), a.group, grp, D) + part_unit_stride(a.group) * (blk / 2);
  const f32x2* lp = reinterpret_cast<const f32x2*>(a.plan.l_part) + row0;
  f32x2 ml[kMergeBatch];
  u32x4 ov[kMergeBatch];
#pragma unroll
  for (int k = 0; k < kMergeBatch; ++k) {
    if (k < mh.nparts) {
      ml[k] = lp[k * stride];
      ov[k] = *reinterpret_cast<const u32x4*>(op + k * stride * D);
    } else {
      ml[k] = f32x2{kNegBig, 0.f};
      ov[k] = u32x4{0u, 0u, 0u, 0u};
    }
  }
  float mx = kNegBig;
#pragma unroll
  for (int k = 0; k < kMergeBatch; ++k) mx = fmaxf(mx, ml[k][0]);
  for (int k = kMergeBatch; k < mh.nparts; ++k) mx = fmaxf(mx, lp[k * stride][0]);
  float z = 0.f;
  f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
  // Part k weighs 2^(m_k - mx) l_k: its values are already divided by l_k.
#pragma unroll
  for (int k = 0; k < kMergeBatch; ++k) {
    const float wl = fast_exp2(ml[k][0] - mx) * ml[k][1];  // 0 for unused slots and for pieces that saw no key
    z += wl;
    acc0 += wl * unpack_bf16x4(ov[k][0], ov[k][1]);
    acc1 += wl * unpack_bf16x4(ov[k][2], ov[k][3]);
  }
  for (int k = kMergeBatch; k < mh.nparts; ++k) {
    const f32x2 x = lp[k * stride];
    const float wl = fast_exp2(x[0] - mx) * x[1];
    const u32x4 v = *reinterpret_cast<const u32x4*>(op + k * stride * D);
    z += wl;
    acc0 += wl * unpack_bf16x4(v[0], v[1]);
    acc1 += wl * unpack_bf16x4(v[2], v[3]);
  }
  const float inv = 1.0f / z;
  uint16_t* out = a.o + (size_t(tok) * a.hq + qh) * D + 16 * blk + 4 * grp;
  *reinterpret_cast<u32x2*>(out) = u32x2{pack_bf16(acc0[0] * inv, acc0[1] * inv), pack_bf16(acc0[2] * inv, acc0[3] * inv)};
  *reinterpret_cast<u32x2*>(out + 16) =
      u32x2{pack_bf16(acc1[0] * inv, acc1[1] * inv), pack_bf16(acc1[2] * inv, acc1[3] * inv)};
  if (a.lse && sl == 0) a.lse[size_t(tok) * a.hq + qh] = (mx + log2f(z)) * kLn2;
  if constexpr (F) {
#pragma unroll
    for (int i = 0; i < kAppendPerThread; ++i)
      if (app_dst[i]) *reinterpret_cast<u32x4*>(app_dst[i]) = app_val[i];
  }
}

template <int D>
__global__ __launch_bounds__(256) void merge_states_kernel(const float* o_parts, const float* lse_parts, int nparts,
                                                           int rows, uint16_t* o, float* lse) {
  constexpr int SL = D / 8;
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= rows * SL) return;
  const int x = t / SL, sl = t - x * SL;
  merge_row8(o_parts + size_t(x) * D + sl * 8, size_t(rows) * D, lse_parts + x, size_t(rows), nparts,
             o + size_t(x) * D + sl * 8, (lse && sl == 0) ? lse + x : nullptr);
}

// One thread per 16-byte chunk of a new token's K or V row.
template <int D>
__global__ __launch_bounds__(256) void append_kernel(const uint16_t* k_new, const uint16_t* v_new, uint16_t* kpool,
                                                     uint16_t* vpool, const int32_t* tok_slot, int tokens, int hkv) {
  constexpr int CPR = D / 8;  // chunks per (token, head)
  const size_t per = size_t(tokens) * hkv * CPR;
  const size_t idx = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= 2 * per) return;
  const bool is_v = idx >= per;
  const size_t e = is_v ? idx - per : idx;
  const int c = int(e % CPR);
  const size_t th = e / CPR;
  const int hh = int(th % hkv);
  const int t = int(th / hkv);
  const int slot = tok_slot[t];
  const size_t dst = ((size_t(slot >> 4) * hkv + hh) * 16 + (slot & 15)) * D + 8 * c;
  const size_t src = (size_t(t) * hkv + hh) * D + 8 * c;
  const uint16_t* s = is_v ? v_new : k_new;
  uint16_t* d = is_v ? vpool : kpool;
  *reinterpret_cast<u32x4*>(d + dst) = *reinterpret_cast<const u32x4*>(s + src);
}

// grid (chunks of a page, pages, 2 for K/V); pairs[2i] = dst page, pairs[2i+1] = src page.
__global__ __launch_bounds__(256) void page_copy_kernel(const u32x4* src_k, const u32x4* src_v, u32x4* dst_k,
                                                        u32x4* dst_v, const int32_t* pairs, size_t page_vecs) {
  const size_t v = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (v >= page_vecs) return;
  const int i = blockIdx.y;
  const size_t dp = size_t(pairs[2 * i]), sp = size_t(pairs[2 * i + 1]);
  if (blockIdx.z == 0)
    dst_k[dp * page_vecs + v] = src_k[sp * page_vecs + v];
  else
    dst_v[dp * page_vecs + v] = src_v[sp * page_vecs + v];
}

static int hip_fail(hipError_t e, const char* what) {
  return fail(PFX_EHIP, "%s: %s", what, hipGetErrorString(e));
}

static int check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? PFX_OK : hip_fail(e, what);
}

static int check_pool_matches(const pfx_pool* pool, const pfx_plan* p, const char* who) {
  if (!pool) return fail(PFX_EINVAL, "%s: pool is NULL", who);
  if (!p) return fail(PFX_EINVAL, "%s: plan is NULL", who);
  if (pool->page_size != PFX_PAGE_SIZE || pool->num_kv_heads != p->hkv || pool->head_dim != p->d ||
      pool->num_pages != p->num_pages)
    return fail(PFX_EINVAL, "%s: pool shape differs from the one the plan was built for", who);
  if (!pool->k_pages || !pool->v_pages) return fail(PFX_EINVAL, "%s: pool pointers are NULL", who);
  if (!p->dev_ws) return fail(PFX_EINVAL, "%s: plan has not been uploaded", who);
  return PFX_OK;
}

// The decode launch alone: wide prefix blocks (if any) and the pieces.
template <int D>
static void launch_decode(const AttnArgs& a, const pfx_plan* p, hipStream_t s) {
  const int S = std::min<int>(a.num_workers, p->num_segs);
  const dim3 grid(p->num_wide + S);
  if (p->decode_engine == PFX_DECODE_VALU) {
    if (a.fuse_append) hipLaunchKernelGGL((decode_kernel<D, true, false, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((decode_kernel<D, false, false, true>), grid, dim3(256), 0, s, a);
  } else if (a.fuse_append) {
    if (p->num_wide) hipLaunchKernelGGL((decode_kernel<D, true, true, false>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((decode_kernel<D, true, false, false>), grid, dim3(256), 0, s, a);
  } else {
    if (p->num_wide) hipLaunchKernelGGL((decode_kernel<D, false, true, false>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((decode_kernel<D, false, false, false>), grid, dim3(256), 0, s, a);
  }
}

template <int D>
static void launch_all(AttnArgs a, const pfx_plan* p, hipStream_t s) {
  if (p->num_items > 0 && p->num_segs > 0 && p->decode_engine == PFX_DECODE_MFMA && !a.fuse_append) {
    // A mixed batch in one launch: the extend blocks and the wide prefix
    // blocks lead the grid (the same block routine as the extend launch, at
    // the same block indices, so their XCD grouping holds), and the decode
    // pieces follow, taking compute units as the extend blocks retire
    // instead of waiting for the last of them.
    AttnArgs m = a;
    m.num_wide = p->num_items + p->num_wide;
    m.wide_first = 0;
    const int S = std::min<int>(a.num_workers, p->num_segs);
    hipLaunchKernelGGL((decode_kernel<D, false, true, false>), dim3(m.num_wide + S), dim3(256), 0, s, m);
  } else {
    if (p->num_items > 0) hipLaunchKernelGGL((extend_kernel<D>), dim3(p->num_items), dim3(256), 0, s, a);
    if (p->num_segs > 0 || p->num_wide > 0) launch_decode<D>(a, p, s);
  }
  const int n_tok = static_cast<int>(p->merge_tok.size());
  if (n_tok) {
    // Workgroups of 128 threads: a decode-8B merge (32768 threads) then
    // spreads over every compute unit instead of half of them.
    constexpr int kMergeThreads = 128;
    const size_t threads = size_t(n_tok) * p->hq * (D / 8);
    const dim3 grid((threads + kMergeThreads - 1) / kMergeThreads);
    if (a.fuse_append)
      hipLaunchKernelGGL((merge_rows_kernel<D, true>), grid, dim3(kMergeThreads), 0, s, a, n_tok);
    else
      hipLaunchKernelGGL((merge_rows_kernel<D, false>), grid, dim3(kMergeThreads), 0, s, a, n_tok);
  }
}

}  // namespace pfx

using namespace pfx;

extern "C" int pfx_plan_upload(pfx_plan* p, void* ws, size_t bytes, void* stream) {
  if (!p || !ws) return fail(PFX_EINVAL, "pfx_plan_upload: NULL argument");
  if (reinterpret_cast<uintptr_t>(ws) % 256) return fail(PFX_EINVAL, "pfx_plan_upload: workspace not 256-byte aligned");
  if (bytes < p->total_bytes)
    return fail(PFX_ENOMEM, "pfx_plan_upload: workspace has %zu bytes, plan needs %zu", bytes, p->total_bytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (p->blob_bytes) {
    hipError_t e = hipMemcpyAsync(ws, p->blob.data(), p->blob_bytes, hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return hip_fail(e, "pfx_plan_upload: hipMemcpyAsync");
  }
  p->dev_ws = ws;
  p->dev_ws_bytes = bytes;
  return PFX_OK;
}

// The KV append of a plan whose tables sit at dp (validated by the caller).
static int launch_append(const pfx_pool* pool, const pfx_plan* p, const DevPlan& dp, const void* k_new,
                         const void* v_new, hipStream_t s, const char* who) {
  const size_t total = 2 * size_t(p->num_tokens) * p->hkv * (p->d / 8);
  const dim3 grid((total + 255) / 256);
  auto kn = static_cast<const uint16_t*>(k_new);
  auto vn = static_cast<const uint16_t*>(v_new);
  auto kp = static_cast<uint16_t*>(pool->k_pages);
  auto vp = static_cast<uint16_t*>(pool->v_pages);
  if (p->d == 128)
    hipLaunchKernelGGL(append_kernel<128>, grid, dim3(256), 0, s, kn, vn, kp, vp, dp.tok_slot, p->num_tokens, p->hkv);
  else
    hipLaunchKernelGGL(append_kernel<64>, grid, dim3(256), 0, s, kn, vn, kp, vp, dp.tok_slot, p->num_tokens, p->hkv);
  return check_launch(who);
}

// The attention launches of a plan whose tables and partial states sit at
// dp (validated by the caller).
static int launch_attention(const pfx_pool* pool, const pfx_plan* p, const DevPlan& dp, const void* q, void* o,
                            float* lse, float sm_scale, hipStream_t s, const char* who, const void* k_new = nullptr,
                            const void* v_new = nullptr) {
  if (!(sm_scale > 0.f)) sm_scale = 1.0f / sqrtf(float(p->d));
  AttnArgs a;
  a.k_new = static_cast<const uint16_t*>(k_new);
  a.v_new = static_cast<const uint16_t*>(v_new);
  a.fuse_append = k_new != nullptr;
  a.kpool = static_cast<const uint16_t*>(pool->k_pages);
  a.vpool = static_cast<const uint16_t*>(pool->v_pages);
  a.q = static_cast<const uint16_t*>(q);
  a.o = static_cast<uint16_t*>(o);
  a.lse = lse;
  a.plan = dp;
  a.hq = p->hq;
  a.hkv = p->hkv;
  a.group = p->group;
  a.group_shift = __builtin_ctz(static_cast<unsigned>(p->group));
  a.scale_log2 = sm_scale * kLog2e;
  a.num_pieces = p->num_segs;
  // By default one workgroup per piece: the dispatcher hands them out as
  // compute units free up (two fit on one), in list order, longest first.
  a.num_workers = p->decode_workers > 0 ? p->decode_workers : p->num_segs;
  a.num_wide = p->num_wide;
  a.wide_first = p->num_items;
  a.merge_parts = p->merge_parts;
  a.merge_tok_is_row = p->merge_tok_is_row;
  if (p->d == 128) launch_all<128>(a, p, s); else launch_all<64>(a, p, s);
  return check_launch(who);
}

extern "C" int pfx_append_kv(const pfx_pool* pool, const pfx_plan* p, const void* k_new, const void* v_new,
                             void* stream) {
  int rc = check_pool_matches(pool, p, "pfx_append_kv");
  if (rc) return rc;
  if (p->num_tokens == 0) return PFX_OK;
  if (!k_new || !v_new) return fail(PFX_EINVAL, "pfx_append_kv: k_new or v_new is NULL");
  return launch_append(pool, p, dev_plan(p), k_new, v_new, static_cast<hipStream_t>(stream), "pfx_append_kv");
}

extern "C" int pfx_attention(const pfx_pool* pool, const pfx_plan* p, const void* q, void* o, float* lse,
                             float sm_scale, void* stream) {
  int rc = check_pool_matches(pool, p, "pfx_attention");
  if (rc) return rc;
  if (p->num_items == 0 && p->num_segs == 0 && p->num_wide == 0) return PFX_OK;
  if (!q || !o) return fail(PFX_EINVAL, "pfx_attention: q or o is NULL");
  return launch_attention(pool, p, dev_plan(p), q, o, lse, sm_scale, static_cast<hipStream_t>(stream),
                          "pfx_attention");
}

// The append and the attention of one step in the fewest launches: with no
// extend blocks (which read each other's new tokens) the decode pieces take
// their new tokens straight from k_new / v_new and write them into the pool
// themselves; otherwise the append kernel runs first.
static int step_launches(const pfx_pool* pool, const pfx_plan* p, const DevPlan& dp, const void* k_new,
                         const void* v_new, const void* q, void* o, float* lse, float sm_scale, hipStream_t s,
                         const char* who) {
  const bool attend = p->num_items > 0 || p->num_segs > 0 || p->num_wide > 0;
  if (p->num_tokens > 0 && (p->num_items > 0 || !attend)) {
    int rc = launch_append(pool, p, dp, k_new, v_new, s, who);
    if (rc || !attend) return rc;
    return launch_attention(pool, p, dp, q, o, lse, sm_scale, s, who);
  }
  if (!attend) return PFX_OK;
  return launch_attention(pool, p, dp, q, o, lse, sm_scale, s, who, k_new, v_new);
}

extern "C" int pfx_step(const pfx_pool* pool, const pfx_plan* p, const void* k_new, const void* v_new,
                        const void* q, void* o, float* lse, float sm_scale, void* stream) {
  int rc = check_pool_matches(pool, p, "pfx_step");
  if (rc) return rc;
  if (p->num_tokens > 0 && (!k_new || !v_new)) return fail(PFX_EINVAL, "pfx_step: k_new or v_new is NULL");
  if ((p->num_items > 0 || p->num_segs > 0 || p->num_wide > 0) && (!q || !o))
    return fail(PFX_EINVAL, "pfx_step: q or o is NULL");
  return step_launches(pool, p, dev_plan(p), k_new, v_new, q, o, lse, sm_scale, static_cast<hipStream_t>(stream),
                       "pfx_step");
}

// ---------------------------------------------------------------------------
// Allocation-free variant: the plan's tables and the decode pieces' partial
// states live in one file-scope device array instead of a caller workspace.
// Each GPU holds its own copy until the process ends; host code reaches it
// only through the address hipGetSymbolAddress returns for the current
// device (the array's name is a host-side stand-in, not a device address).
// ---------------------------------------------------------------------------
namespace pfx {
constexpr size_t kScratchBytes = PFX_NOALLOC_MAX_WORKSPACE;
constexpr int kMaxScratchDevices = 64;
}  // namespace pfx

static __device__ __align__(256) unsigned char scratch[pfx::kScratchBytes];

namespace pfx {
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxScratchDevices];

// Device address of `scratch` on the current device, looked up on the first
// call on each device and kept.
static int scratch_address(void** out, const char* who) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, who);
  if (dev < 0 || dev >= kMaxScratchDevices) return fail(PFX_EINVAL, "%s: device %d out of range", who, dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!ptr || reinterpret_cast<uintptr_t>(ptr) % 256)
      return fail(PFX_EHIP, "%s: scratch address %p is not 256-byte aligned", who, ptr);
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return PFX_OK;
}
}  // namespace pfx

extern "C" int pfx_attention_noalloc(const pfx_pool* pool, const pfx_plan* p, const void* k_new,
                                     const void* v_new, const void* q, void* o, float* lse, float sm_scale,
                                     void* stream) {
  const char* who = "pfx_attention_noalloc";
  if (!pool) return fail(PFX_EINVAL, "%s: pool is NULL", who);
  if (!p) return fail(PFX_EINVAL, "%s: plan is NULL", who);
  if (pool->page_size != PFX_PAGE_SIZE || pool->num_kv_heads != p->hkv || pool->head_dim != p->d ||
      pool->num_pages != p->num_pages)
    return fail(PFX_EINVAL, "%s: pool shape differs from the one the plan was built for", who);
  if (!pool->k_pages || !pool->v_pages) return fail(PFX_EINVAL, "%s: pool pointers are NULL", who);
  if ((k_new == nullptr) != (v_new == nullptr))
    return fail(PFX_EINVAL, "%s: k_new and v_new must both be given or both be NULL", who);
  const bool attend = p->num_items > 0 || p->num_segs > 0 || p->num_wide > 0;
  if (attend && (!q || !o)) return fail(PFX_EINVAL, "%s: q or o is NULL", who);
  if (p->total_bytes > kScratchBytes)
    return fail(PFX_ENOMEM, "%s: the plan needs %zu bytes of workspace, the static scratch holds %zu", who,
                p->total_bytes, kScratchBytes);
  const bool append = k_new != nullptr && p->num_tokens > 0;
  if (!append && !attend) return PFX_OK;
  void* ws = nullptr;
  int rc = scratch_address(&ws, who);
  if (rc) return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  // The tables, stream-ordered after any earlier call's kernels that read
  // them; the partial states need no clearing (every slot is written by its
  // piece before the merge reads it).
  if (p->blob_bytes) {
    hipError_t e = hipMemcpyAsync(ws, p->blob.data(), p->blob_bytes, hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return hip_fail(e, "pfx_attention_noalloc: hipMemcpyAsync");
  }
  const DevPlan dp = dev_plan(p, ws);
  if (append) return step_launches(pool, p, dp, k_new, v_new, q, o, lse, sm_scale, s, who);
  return launch_attention(pool, p, dp, q, o, lse, sm_scale, s, who);
}

extern "C" int pfx_merge_states(const float* o_parts, const float* lse_parts, int32_t num_parts, int32_t rows,
                                int32_t head_dim, void* o, float* lse, void* stream) {
  if (!o_parts || !lse_parts || !o) return fail(PFX_EINVAL, "pfx_merge_states: NULL argument");
  if (head_dim != 64 && head_dim != 128) return fail(PFX_EUNSUPPORTED, "pfx_merge_states: head_dim %d", head_dim);
  if (num_parts < 1 || num_parts > 4096) return fail(PFX_ERANGE, "pfx_merge_states: num_parts %d", num_parts);
  if (rows < 0) return fail(PFX_ERANGE, "pfx_merge_states: rows %d", rows);
  if (rows == 0) return PFX_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t threads = size_t(rows) * (head_dim / 8);
  const dim3 grid((threads + 255) / 256);
  if (head_dim == 128)
    hipLaunchKernelGGL(merge_states_kernel<128>, grid, dim3(256), 0, s, o_parts, lse_parts, num_parts, rows,
                       static_cast<uint16_t*>(o), lse);
  else
    hipLaunchKernelGGL(merge_states_kernel<64>, grid, dim3(256), 0, s, o_parts, lse_parts, num_parts, rows,
                       static_cast<uint16_t*>(o), lse);
  return check_launch("pfx_merge_states");
}

extern "C" size_t pfx_page_copy_workspace_bytes(int32_t n) { return n <= 0 ? 256 : (size_t(n) * 8 + 255) & ~size_t(255); }

extern "C" int pfx_page_copy(const pfx_pool* dst, const pfx_pool* src, const int32_t* dst_pages,
                             const int32_t* src_pages, int32_t n, void* ws, size_t ws_bytes, void* stream) {
  if (!dst || !src) return fail(PFX_EINVAL, "pfx_page_copy: pool descriptor is NULL");
  if (n < 0) return fail(PFX_ERANGE, "pfx_page_copy: n %d < 0", n);
  if (n == 0) return PFX_OK;
  if (!dst_pages || !src_pages || !ws) return fail(PFX_EINVAL, "pfx_page_copy: NULL argument");
  if (dst->page_size != PFX_PAGE_SIZE || src->page_size != PFX_PAGE_SIZE)
    return fail(PFX_EUNSUPPORTED, "pfx_page_copy: page_size must be %d", PFX_PAGE_SIZE);
  if (dst->num_kv_heads != src->num_kv_heads || dst->head_dim != src->head_dim || dst->num_kv_heads < 1 ||
      dst->head_dim < 8 || dst->head_dim % 8)
    return fail(PFX_EINVAL, "pfx_page_copy: source and destination page formats differ");
  if (!dst->k_pages || !dst->v_pages || !src->k_pages || !src->v_pages)
    return fail(PFX_EINVAL, "pfx_page_copy: page pointers are NULL");
  if (reinterpret_cast<uintptr_t>(ws) % 256) return fail(PFX_EINVAL, "pfx_page_copy: workspace not 256-byte aligned");
  if (ws_bytes < pfx_page_copy_workspace_bytes(n))
    return fail(PFX_ENOMEM, "pfx_page_copy: workspace has %zu bytes, needs %zu", ws_bytes,
                pfx_page_copy_workspace_bytes(n));
  std::vector<int32_t> pairs(2 * size_t(n));
  std::vector<uint8_t> seen(dst->num_pages, 0);
  for (int32_t i = 0; i < n; ++i) {
    if (dst_pages[i] < 0 || dst_pages[i] >= dst->num_pages)
      return fail(PFX_ERANGE, "pfx_page_copy: dst_pages[%d] = %d outside [0, %d)", i, dst_pages[i], dst->num_pages);
    if (src_pages[i] < 0 || src_pages[i] >= src->num_pages)
      return fail(PFX_ERANGE, "pfx_page_copy: src_pages[%d] = %d outside [0, %d)", i, src_pages[i], src->num_pages);
    if (seen[dst_pages[i]]) return fail(PFX_EINVAL, "pfx_page_copy: destination page %d repeated", dst_pages[i]);
    seen[dst_pages[i]] = 1;
    pairs[2 * i] = dst_pages[i];
    pairs[2 * i + 1] = src_pages[i];
  }
  // Every page array must be device memory or pinned host memory (the
  // kernel would fault on pageable host memory).
  for (const void* ptr : {dst->k_pages, dst->v_pages, src->k_pages, src->v_pages}) {
    hipPointerAttribute_t at;
    if (hipPointerGetAttributes(&at, ptr) != hipSuccess) {
      (void)hipGetLastError();
      return fail(PFX_EINVAL, "pfx_page_copy: a page pointer is neither device nor pinned host memory");
    }
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipMemcpyAsync(ws, pairs.data(), pairs.size() * 4, hipMemcpyHostToDevice, s);
  if (e != hipSuccess) return hip_fail(e, "pfx_page_copy: hipMemcpyAsync");
  const size_t page_bytes = size_t(dst->num_kv_heads) * PFX_PAGE_SIZE * dst->head_dim * 2;
  const size_t page_vecs = page_bytes / 16;
  // gridDim.y is limited to 65535: launch the page list in slices.
  for (int32_t at = 0; at < n; at += 65535) {
    const int32_t cnt = std::min<int32_t>(65535, n - at);
    const dim3 grid((page_vecs + 255) / 256, cnt, 2);
    hipLaunchKernelGGL(page_copy_kernel, grid, dim3(256), 0, s, static_cast<const u32x4*>(src->k_pages),
                       static_cast<const u32x4*>(src->v_pages), static_cast<u32x4*>(dst->k_pages),
                       static_cast<u32x4*>(dst->v_pages), static_cast<const int32_t*>(ws) + 2 * size_t(at),
                       page_vecs);
    int rc = check_launch("pfx_page_copy");
    if (rc) return rc;
  }
  return PFX_OK;
}

extern "C" int pfx_sync_check(void* stream) {
  hipError_t e = hipStreamSynchronize(static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "pfx_sync_check");
  e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "pfx_sync_check");
  return PFX_OK;
}
