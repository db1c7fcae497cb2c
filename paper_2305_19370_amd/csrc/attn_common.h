// Device helpers shared by the attention kernels: the LDS tile layout, the ring of
// direct global->LDS copies, MFMA fragment reads (plain and transposed), and the
// workgroup -> (head, block) mapping.
#pragma once

#include <type_traits>

#include "common.h"
#include "internal.h"

namespace bpt {

static constexpr float LOG2E = 1.4426950408889634f;
static constexpr float LN2 = 0.6931471805599453f;
static constexpr float NEG_INF = -__builtin_inff();

// Row-major LDS tile: 64 token rows of DH bf16 features. The pitch (DH*2 + 48 bytes
// for DH = 128, DH*2 + 16 for DH = 64) is an odd multiple of 16 bytes, so the 16 rows
// of a 16-byte fragment read start in distinct bank groups, and it spreads the four
// 32-byte row pieces of a transposed read over distinct banks as well. Every fragment
// address is a per-lane base plus a compile-time offset.
template <int DH>
struct RmTile {
  static constexpr int PITCH = DH == 128 ? 304 : 144;
  static constexpr int SLOTS = PITCH / 16;            // 16-byte slots per row
  static constexpr int BYTES = 64 * PITCH;
  static constexpr int BLOCKS = BYTES / 1024;         // 1 KiB blocks (one wave-wide copy each)
  static_assert(DH == 64 || DH == 128, "head dim");
  static_assert(BYTES % 1024 == 0, "tile must be whole 1 KiB blocks");
};

BPT_DEV u32x4 ld16(const void* p) { return *(const u32x4*)p; }

// Force the completion of earlier global loads into v before the code that follows
// (the compiler would otherwise place its own wait at the first use, inside a loop).
BPT_DEV void settle(const bf16x8& v) { asm volatile("" ::"v"(v)); }
BPT_DEV void settle(float v) { asm volatile("" ::"v"(v)); }

// Direct global -> LDS copy: every lane of the wave fetches 16 (or 4) bytes from a
// wave-uniform base address (SGPR pair) plus its own 32-bit byte offset; lane l's
// bytes land at lds_block + 16 l (4 l). Inline assembly rather than the builtin: the
// compiler's counter tracking treats the builtin as a pending FLAT access and then
// drains every later LDS-read wait to zero. Completion is waited for by hand
// (wait_vmcnt); M0 is not otherwise used in these kernels.
BPT_DEV uint32_t lds_addr(const char* p) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(__attribute__((address_space(3))) const char*)p);
}
BPT_DEV void dma16s(const void* sbase, uint32_t voff, char* lds_block) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(voff), "s"(sbase), "s"(lds_addr(lds_block)) : "memory");
}
BPT_DEV void dma4s(const void* sbase, uint32_t voff, char* lds_block) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1"
               :: "v"(voff), "s"(sbase), "s"(lds_addr(lds_block)) : "memory");
}
template <int N> BPT_DEV void wait_vmcnt() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }

BPT_DEV float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }   // v_exp_f32; exp2(-inf) = 0

// Copies of stages made of two row-major tiles (rows row0 .. row0+63 of two tensors).
// The 2 * BLOCKS copy blocks of a stage are dealt to the NW waves round robin; every
// wave issues the same number DPW (surplus slots repeat the last block, which writes
// identical bytes), so a count of outstanding copies is the same on every wave. Pad
// slots re-fetch a data chunk of the same row and are never read.
template <int DH, int NW = 4>
struct Ring2 {
  static constexpr int BL = RmTile<DH>::BLOCKS, NB = 2 * BL, DPW = (NB + NW - 1) / NW;
};

template <int DH, int NW>
BPT_DEV int ring_block(int wave, int i) {
  const int b = wave + NW * i;
  return b < Ring2<DH, NW>::NB ? b : Ring2<DH, NW>::NB - 1;
}

// Issue this wave's copies of one stage: rows row0 .. row0+63 of src0 into the first
// tile, rows row1 .. row1+63 of src1 into the second. Rows past last_row are clamped
// to it (the kernels mask them); row0, row1 <= last_row.
template <int DH, int NW = 4>
BPT_DEV void ring_issue(char* stage, const bf16* src0, int ld0, int row0, const bf16* src1, int ld1, int row1,
                        int last_row, int wave, int lane) {
  using T = RmTile<DH>;
  const bf16* org0 = src0 + (int64_t)row0 * ld0;
  const bf16* org1 = src1 + (int64_t)row1 * ld1;
  const int lim0 = last_row - row0 < 63 ? last_row - row0 : 63;
  const int lim1 = last_row - row1 < 63 ? last_row - row1 : 63;
  // recomputed at every call: hoisting the offsets out of the tile loop would cost
  // one register each for the whole kernel
  asm volatile("" : "+v"(lane));
#pragma unroll
  for (int i = 0; i < Ring2<DH, NW>::DPW; ++i) {
    const int b = ring_block<DH, NW>(wave, i), t = b >= T::BLOCKS, blk = b - t * T::BLOCKS;
    const int slot = blk * 64 + lane, col = slot % T::SLOTS, lim = t ? lim1 : lim0;
    int row = slot / T::SLOTS;
    row = row < lim ? row : lim;
    const uint32_t off = 2u * (uint32_t)(row * (t ? ld1 : ld0) + (col < DH / 8 ? col : 0) * 8);
    dma16s(t ? org1 : org0, off, stage + t * T::BYTES + blk * 1024);
  }
}

// The per-lane byte offsets of ring_issue for a stage whose 64 rows all exist
// (row0 + 63 <= last_row), computed once per kernel: they depend only on the lane,
// the wave and the two row strides.
template <int DH, int NW>
struct RingOff {
  uint32_t o[Ring2<DH, NW>::DPW];
};

template <int DH, int NW>
BPT_DEV RingOff<DH, NW> ring_offsets(int ld0, int ld1, int wave, int lane) {
  using T = RmTile<DH>;
  RingOff<DH, NW> r;
#pragma unroll
  for (int i = 0; i < Ring2<DH, NW>::DPW; ++i) {
    const int b = ring_block<DH, NW>(wave, i), t = b >= T::BLOCKS, blk = b - t * T::BLOCKS;
    const int slot = blk * 64 + lane, col = slot % T::SLOTS, row = slot / T::SLOTS;
    r.o[i] = 2u * (uint32_t)(row * (t ? ld1 : ld0) + (col < DH / 8 ? col : 0) * 8);
  }
  return r;
}

// ring_issue for a stage whose rows all exist, with precomputed offsets.
template <int DH, int NW>
BPT_DEV void ring_issue_full(char* stage, const bf16* src0, int ld0, int row0, const bf16* src1, int ld1, int row1,
                             const RingOff<DH, NW>& r, int wave) {
  using T = RmTile<DH>;
  const bf16* org0 = src0 + (int64_t)row0 * ld0;
  const bf16* org1 = src1 + (int64_t)row1 * ld1;
#pragma unroll
  for (int i = 0; i < Ring2<DH, NW>::DPW; ++i) {
    const int b = ring_block<DH, NW>(wave, i), t = b >= T::BLOCKS, blk = b - t * T::BLOCKS;
    dma16s(t ? org1 : org0, r.o[i], stage + t * T::BYTES + blk * 1024);
  }
}

// A-operand fragment with tile rows as MFMA rows: lane l reads row (row0 + l%32),
// features 8*kc' .. 8*kc'+7 where kc' = kc + l/32 (kc even).
template <int DH>
BPT_DEV bf16x8 frag_rows(const char* tile, int row0, int kc, int lane) {
  return *(const bf16x8*)(tile + (row0 + (lane & 31)) * RmTile<DH>::PITCH + (kc + (lane >> 5)) * 16);
}

typedef __attribute__((__vector_size__(4 * sizeof(short)))) short s16x4;
typedef __attribute__((__vector_size__(8 * sizeof(short)))) short s16x8;

// A-operand fragment of the transposed tile for a contraction over 16 tile rows:
// lane l supplies feature d0 + l%32 at rows tok0 + 4*(l/32) + {0..3} and
// tok0 + 8 + 4*(l/32) + {0..3}, the order in which an MFMA accumulator hands its rows
// to the next MFMA as a B operand. Two ds_read_b64_tr_b16: inside each group of 16
// lanes, lane m addresses 4 features of one row (row m/4, features 4*(m%4)..), and
// the instruction returns to lane m feature m of rows 0..3 of the group.
template <int DH>
BPT_DEV bf16x8 frag_tr(const char* tile, int tok0, int d0, int lane) {
  const int g = lane >> 4, m = lane & 15;
  const char* p = tile + (tok0 + 4 * (g >> 1) + (m >> 2)) * RmTile<DH>::PITCH + (d0 + 16 * (g & 1) + 4 * (m & 3)) * 2;
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
  const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)p);
  const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p + 8 * RmTile<DH>::PITCH));
  const s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8, v);
}

// max(v[l], v[l ^ 32]) for every lane l, without LDS.
BPT_DEV float max_halves(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
BPT_DEV float sum_halves(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Registers 8*hf .. 8*hf+7 of an accumulator as a bf16 B operand.
BPT_DEV bf16x8 acc_to_b(const f32x16& s, int hf) {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = (bf16)s[8 * hf + i];
  return r;
}

// Row of accumulator register r for lane `lane` inside a 32x32 tile.
BPT_DEV int acc_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

// Workgroup id -> (head instance hh in [0, NH), block index blk). Workgroup i runs
// on XCD i % 8 and every XCD has its own L2; when NH is a multiple of 8, all blocks of
// a head run on one XCD, so the blocks that stream the same K/V (or Q/dO) tiles share
// that L2. Block 0 of every head is dispatched first.
BPT_DEV void xcd_map(int id, int NH, int& hh, int& blk) {
  if ((NH & 7) == 0) {
    const int x = id & 7, k = id >> 3, hp = NH >> 3;
    hh = x + 8 * (k % hp);
    blk = k / hp;
  } else {
    hh = id % NH;
    blk = id / NH;
  }
}

// xcd_map for kernels whose heads have many blocks (nblk >= 128): when NH is a multiple
// of 8, XCD x serves its heads x, x + 8, ... in turns of 32 consecutive blocks (blocks
// 0 .. 31 of each of its heads, then blocks 32 .. 63 of each, ...; the last turn may be
// shorter). The 32 workgroups an XCD holds at once then mostly belong to one head and
// walk the same tiles together, so that fewer of the tiles they stream are fetched
// from HBM again, while the turns still start the blocks with the most work first.
// With fewer blocks per head the turns would mix heavy and light blocks within one
// generation of workgroups, and xcd_map's order is kept.
BPT_DEV void xcd_map_heads(int id, int NH, int nblk, int& hh, int& blk) {
  constexpr int CHUNK = 32;
  if ((NH & 7) != 0 || nblk < 4 * CHUNK) {
    xcd_map(id, NH, hh, blk);
    return;
  }
  const int x = id & 7, k = id >> 3, hp = NH >> 3;
  const int full = nblk / CHUNK;                // turns of a whole chunk per head
  int turn = k / (hp * CHUNK), c = CHUNK;
  if (turn >= full) {                           // the last, shorter turn
    turn = full;
    c = nblk - full * CHUNK;
  }
  const int r = k - turn * hp * CHUNK;
  hh = x + 8 * (r / c);
  blk = turn * CHUNK + r % c;
}

template <typename K>
static hipError_t set_lds(K kern, int bytes) {
  return hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
}

}  // namespace bpt
