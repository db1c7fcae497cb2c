// Device helpers shared by the attention kernels (LDS tile layouts, direct
// global->LDS copies, MFMA fragment plumbing).
#pragma once

#include <type_traits>

#include "common.h"
#include "internal.h"

namespace bpt {

static constexpr float LOG2E = 1.4426950408889634f;
static constexpr float NEG_INF = -__builtin_inff();

// LDS tile layouts. Rows are padded by one 16-byte slot so that the 32 rows a
// fragment read touches start in different banks, and every fragment address is
// one per-lane base plus a compile-time offset.
//  * row-major tile: 64 rows of DH bf16 (DH/8 data slots + 1 pad slot per row);
//  * feature-major tile: DH rows of 64 tokens (8 data slots + 1 pad slot per row).
template <int DH>
struct RmTile {
  static constexpr int SLOTS = DH / 8 + 1;
  static constexpr int PITCH = SLOTS * 16;
  static constexpr int BYTES = 64 * PITCH;
  static constexpr int BLOCKS = BYTES / 1024;        // 1 KB blocks (one wave-wide copy each)
  static_assert(BYTES % 1024 == 0, "tile must be whole 1 KB blocks");
};
template <int DH>
struct FmTile {
  static constexpr int SLOTS = 9;
  static constexpr int PITCH = SLOTS * 16;
  static constexpr int BYTES = DH * PITCH;
  static constexpr int BLOCKS = BYTES / 1024;
  static_assert(BYTES % 1024 == 0, "tile must be whole 1 KB blocks");
};

// byte offset of 16-byte chunk kc of row `row` in a row-major tile
template <int DH>
BPT_DEV int rm_addr(int row, int kc) { return row * RmTile<DH>::PITCH + kc * 16; }

BPT_DEV u32x4 ld16(const void* p) { return *(const u32x4*)p; }

// Direct global -> LDS copy: every lane of the wave fetches 16 bytes from its own
// address; lane l's bytes land at lds_block + 16 * l (lds_block is wave-uniform).
// Inline assembly rather than the builtin: the compiler's counter tracking treats the
// builtin as a pending FLAT access and then drains every later LDS-read wait to zero.
// Completion is waited for by hand (wait_dma); M0 is otherwise unused in these kernels.
BPT_DEV uint32_t lds_addr(const char* p) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(__attribute__((address_space(3))) const char*)p);
}
BPT_DEV void dma16(const void* g, char* lds_block) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :: "v"(g), "s"(lds_addr(lds_block)) : "memory");
}
BPT_DEV void dma4(const void* g, char* lds_block) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off"
               :: "v"(g), "s"(lds_addr(lds_block)) : "memory");
}
BPT_DEV void wait_dma() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

BPT_DEV float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }   // v_exp_f32; exp2(-inf) = 0

// Copies of [64][DH] row-major tiles and [DH][64] feature-major tiles into LDS by the
// 4 waves of a workgroup. Each wave copies the 1 KB blocks wave, wave + 4, ...; the
// per-lane source offsets (in elements, relative to the tile origin) are computed
// once, so a tile's copy only adds its origin. Pad slots re-fetch a data chunk of
// the same row and are never read.
template <int BLOCKS>
struct DmaPlan {
  static constexpr int MAXB = (BLOCKS + 3) / 4;
  int off[MAXB];
};

template <int DH>
BPT_DEV void plan_rows(DmaPlan<RmTile<DH>::BLOCKS>& p, int ld, int wave, int lane) {
  using T = RmTile<DH>;
#pragma unroll
  for (int i = 0; i < p.MAXB; ++i) {
    const int slot = (wave + 4 * i) * 64 + lane;
    const int row = slot / T::SLOTS, col = slot % T::SLOTS;
    p.off[i] = row * ld + (col < DH / 8 ? col : 0) * 8;
  }
}

template <int DH>
BPT_DEV void plan_cols(DmaPlan<FmTile<DH>::BLOCKS>& p, int ld, int wave, int lane) {
  using T = FmTile<DH>;
#pragma unroll
  for (int i = 0; i < p.MAXB; ++i) {
    const int slot = (wave + 4 * i) * 64 + lane;
    const int row = slot / T::SLOTS, col = slot % T::SLOTS;
    p.off[i] = row * ld + (col < 8 ? col : 0) * 8;
  }
}

// Rows row0 .. row0+63 of a row-major tensor; rows past last_row are clamped to it
// (callers mask them).
template <int DH>
BPT_DEV void dma_rows(char* tile, const bf16* base, int64_t ld, int row0, int last_row, int wave, int lane,
                      const DmaPlan<RmTile<DH>::BLOCKS>& p) {
  using T = RmTile<DH>;
  if (row0 + 63 <= last_row) {
    const bf16* org = base + (int64_t)row0 * ld;
#pragma unroll
    for (int i = 0; i < p.MAXB; ++i)
      if (wave + 4 * i < T::BLOCKS) dma16(org + p.off[i], tile + (wave + 4 * i) * 1024);
  } else {
#pragma unroll
    for (int i = 0; i < p.MAXB; ++i) {
      const int blk = wave + 4 * i;
      if (blk >= T::BLOCKS) continue;
      const int slot = blk * 64 + lane;
      const int row = slot / T::SLOTS, col = slot % T::SLOTS;
      int r = row0 + row;
      r = r < last_row ? r : last_row;
      dma16(base + (int64_t)r * ld + (col < DH / 8 ? col : 0) * 8, tile + blk * 1024);
    }
  }
}

// Columns tok0 .. tok0+63 of a feature-major tensor (always in bounds: the padded
// width is a multiple of 64 and the padding is zero).
template <int DH>
BPT_DEV void dma_cols(char* tile, const bf16* base, int tok0, int wave, const DmaPlan<FmTile<DH>::BLOCKS>& p) {
  using T = FmTile<DH>;
  const bf16* org = base + tok0;
#pragma unroll
  for (int i = 0; i < p.MAXB; ++i)
    if (wave + 4 * i < T::BLOCKS) dma16(org + p.off[i], tile + (wave + 4 * i) * 1024);
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

// A-operand fragment for a contraction over 16 tokens starting at `tok0` (a multiple
// of 16) of a feature-major LDS tile: lane l supplies row (row0 + l%32) at tokens
// tok0 + 4*(l/32) + {0..3} and tok0 + 8 + 4*(l/32) + {0..3}, matching the order in
// which an MFMA accumulator hands its rows to the next MFMA as a B operand. The tile
// holds its tokens in tok_perm order, which makes these 8 tokens one 16-byte chunk.
template <int DH>
BPT_DEV bf16x8 fm_frag(const char* tile, int row, int tok0, int lane) {
  return *(const bf16x8*)(tile + row * FmTile<DH>::PITCH + (tok0 + 8 * (lane >> 5)) * 2);
}

// Registers 8*hf .. 8*hf+7 of an accumulator as a bf16 B operand.
BPT_DEV bf16x8 acc_to_b(const f32x16& s, int hf) {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = (bf16)s[8 * hf + i];
  return r;
}

// 32x32x16 bf16 MFMA whose accumulator lives in AGPRs for its whole lifetime (the
// compiler's own placement would copy it through VGPRs every iteration when VGPRs
// are scarce). Five wait states before the MFMA cover a VALU write of its operands.
BPT_DEV void mfma_agpr(f32x16& acc, const bf16x8& a, const bf16x8& b) {
  asm("s_nop 4\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}
// Zero an AGPR accumulator (an MFMA of zero operands with a zero addend), so that
// every definition of the accumulator is an AGPR one. The compiler cannot see the
// MFMA inside the asm, so the asm itself provides the wait states after the VALU
// write of the zero operand.
BPT_DEV void mfma_agpr_zero(f32x16& acc) {
  const bf16x8 z = {};
  asm volatile("s_nop 4\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %1, 0" : "=a"(acc) : "v"(z));
}
// Wait states between the last mfma_agpr on these accumulators and any other use.
BPT_DEV void mfma_agpr_drain(f32x16& a0, f32x16& a1, f32x16& a2, f32x16& a3) {
  asm volatile("s_nop 15\n\ts_nop 15\n\ts_nop 7" : "+a"(a0), "+a"(a1), "+a"(a2), "+a"(a3));
}
BPT_DEV void mfma_agpr_drain(f32x16& a0, f32x16& a1) {
  asm volatile("s_nop 15\n\ts_nop 15\n\ts_nop 7" : "+a"(a0), "+a"(a1));
}

// Row of accumulator register r for lane `lane` inside a 32x32 tile.
BPT_DEV int acc_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }


template <typename K>
static hipError_t set_lds(K kern, int bytes) {
  return hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
}

}  // namespace bpt
