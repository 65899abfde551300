// Diagnostic entry point: one v_mfma_f32_16x16x32_bf16 with the operand and
// result lane layout every kernel of this library assumes --
//   A (16x32): lane l holds A[l % 16][(l / 16) * 8 + e], e = 0..7
//   B (32x16): lane l holds B[(l / 16) * 8 + e][l % 16]
//   C (16x16): lane l holds C[(l / 16) * 4 + i][l % 16], i = 0..3
// so a test can compare C with A @ B.
#include "../../include/war_debug.h"
#include "kernels.h"

namespace {
__global__ void k_mfma_probe(const bf16_t* A, const bf16_t* B, float* Cm) {
  const int l = threadIdx.x;
  const int r = l & 15, g = l >> 4;
  uint4 av = *reinterpret_cast<const uint4*>(A + r * 32 + g * 8);
  uint16_t bv[8];
  for (int e = 0; e < 8; ++e) bv[e] = B[(g * 8 + e) * 16 + r];
  uint4 bp;
  bp.x = bv[0] | (uint32_t(bv[1]) << 16);
  bp.y = bv[2] | (uint32_t(bv[3]) << 16);
  bp.z = bv[4] | (uint32_t(bv[5]) << 16);
  bp.w = bv[6] | (uint32_t(bv[7]) << 16);
  f32x4 c = {0.f, 0.f, 0.f, 0.f};
  c = mfma16(as_bf16x8(av), as_bf16x8(bp), c);
  for (int i = 0; i < 4; ++i) Cm[(g * 4 + i) * 16 + r] = c[i];
}
}  // namespace

extern "C" war_status war_debug_mfma16(const void* A, const void* B, float* C, void* stream) {
  if (!A || !B || !C) return WAR_ERR_INVALID_ARG;
  k_mfma_probe<<<1, 64, 0, static_cast<hipStream_t>(stream)>>>(static_cast<const bf16_t*>(A),
                                                              static_cast<const bf16_t*>(B), C);
  return hipGetLastError() == hipSuccess ? WAR_OK : WAR_ERR_HIP;
}
