// bf16 tile layout in LDS shared by the bf16 and the NV16 attention kernels:
// a K tile [BKV rows][D bf16] and a V^T tile [D rows][BKV bf16], each row cut
// into 16-byte chunks that are XOR-swizzled against LDS bank conflicts.
#pragma once
#include "sage_common.h"

namespace sage {

template <int D, int BKV>
struct Bf16TileT {
  static constexpr int KROW = D * 2;          // bytes per K row
  static constexpr int KCH = KROW / 16;       // chunks per K row (16 or 8)
  static constexpr int VROW = BKV * 2;        // bytes per V^T tile row
  static constexpr int VCH = VROW / 16;       // chunks per V^T tile row (8 or 16)
  static constexpr int K_OFF = 0;
  static constexpr int V_OFF = BKV * KROW;
  static constexpr int BYTES = V_OFF + D * VROW;
  static constexpr int KU = BKV * KCH, VU = D * VCH;
  static constexpr int KPT = KU / 256, VPT = VU / 256;
};

// 16-byte chunk swizzle: lanes of one operand read sit on consecutive rows at
// one chunk; keep 8 (32 banks) or 16 (64 banks) consecutive rows on distinct
// bank groups.  Only row bits 0..4 matter, so a 32-row block offset does not
// change the swizzle.
template <int NCH>
__device__ __forceinline__ int bswz(int row, int ch) {
  if constexpr (NCH == 16) return ch ^ (row & 15);
  else return ch ^ (((row & 31) ^ ((row & 31) >> 3)) & 7);
}

__device__ __forceinline__ v8bf as_bf(const v4i x) { return __builtin_bit_cast(v8bf, x); }

}  // namespace sage
