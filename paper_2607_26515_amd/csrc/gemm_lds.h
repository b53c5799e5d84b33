// LDS-shared FP4 GEMM main loop (the large-tile path of gemm.hip).
//
// A workgroup of WM x WN waves owns a (WM*TM*32) x (WN*TN*32) output tile.  Each K step's
// unique operand data (A fragments of every term, B fragments, and their per-lane scale
// bytes) is fetched once per workgroup: every thread issues the same fixed number of 16-byte
// buffer loads (8-byte for the HiF4 weight records) into a ring of R register stages; one
// stage per K step is written to an LDS double buffer, a barrier publishes it, and the waves
// read their MFMA operands from LDS.  Buffer loads return zero past the end of an operand,
// which covers ragged row and column tiles without branches.
//
// LDS stage layout (bytes): A code planes [term][row tile][plane][64 lanes][16 B],
// B code planes [col tile][...], A scales [term][row tile][64], B scales [col tile][64].
// HiF4 A records (48 B) are stored as three 16-byte planes and HiF4 B records (24 B) as a
// 16-byte and an 8-byte plane, so every LDS read is lane-contiguous (no bank conflicts).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace resq {
namespace lds {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v2i __attribute__((ext_vector_type(2)));

constexpr int32_t kRsrcWord3 = 0x00020000;  // gfx9 raw buffer: 32-bit dwords, no swizzle

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, kRsrcWord3);
}

__device__ __forceinline__ v4i ld16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}
__device__ __forceinline__ v2i ld8(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
}
__device__ __forceinline__ int ld4(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}

// Compile-time geometry of one configuration.
template <int FMT, int WM, int WN, int TM, int TN, int NT>
struct Geo {
  static constexpr int kThreads = 64 * WM * WN;
  static constexpr int MTW = WM * TM;  // row tiles per workgroup
  static constexpr int NTW = WN * TN;  // column tiles per workgroup
  static constexpr int FA = FMT == 0 ? 16 : 48;  // A lane record bytes
  static constexpr int FB = FMT == 0 ? 16 : 24;  // B lane record bytes
  static constexpr int A_FRAG = 64 * FA, B_FRAG = 64 * FB;
  static constexpr int A_BYTES = NT * MTW * A_FRAG;
  static constexpr int B_BYTES = NTW * B_FRAG;
  static constexpr int SA_OFF = A_BYTES + B_BYTES;
  static constexpr int SB_OFF = SA_OFF + NT * MTW * 64;
  static constexpr int STAGE = (SB_OFF + NTW * 64 + 255) / 256 * 256;
  // per-thread load counts (exact: every thread issues the same loads)
  static constexpr int A_CHUNKS = MTW * 64 * (FA / 16);            // 16-byte chunks per term
  static constexpr int A_PER = (A_CHUNKS + kThreads - 1) / kThreads;
  static constexpr int B_CHUNK = FMT == 0 ? 16 : 8;
  static constexpr int B_CHUNKS = NTW * 64 * (FB / B_CHUNK);
  static constexpr int B_PER = (B_CHUNKS + kThreads - 1) / kThreads;
  static constexpr int S_CHUNKS = (NT * MTW + NTW) * 16;           // 4-byte scale chunks
  static constexpr int S_PER = (S_CHUNKS + kThreads - 1) / kThreads;
};

}  // namespace lds
}  // namespace resq
