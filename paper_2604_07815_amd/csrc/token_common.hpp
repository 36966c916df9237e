// Helpers shared by the token-selection kernels.
#pragma once

#include "kernels.hpp"

namespace tls {

// Eight 4-bit codes of one packed dword (byte i = code[2i] | code[2i+1] << 4)
// as floats, in channel order.
__device__ inline void unpack_nibbles8(uint32_t w, float* f) {
  const uint32_t lo = w & 0x0f0f0f0fu, hi = (w >> 4) & 0x0f0f0f0fu;
  f[0] = float(lo & 0xffu);         f[1] = float(hi & 0xffu);
  f[2] = float((lo >> 8) & 0xffu);  f[3] = float((hi >> 8) & 0xffu);
  f[4] = float((lo >> 16) & 0xffu); f[5] = float((hi >> 16) & 0xffu);
  f[6] = float(lo >> 24);           f[7] = float(hi >> 24);
}

// Candidate slot -> token position.  slot = i*B + o addresses offset o of the
// i-th entry of the unit's block list; valid when that entry is a block id
// >= 0 and the token lies below ctx_len.  Ids past the last block set
// TLS_DEVERR_BLOCK_ID and are skipped.
__device__ inline bool slot_token(const int32_t* bl, int K_b, int B, int m, int n, int slot, int* tok,
                                  uint32_t* err) {
  const int i = tok_block(slot, B), o = tok_offset(slot, B);
  if (i >= K_b) return false;
  const int blk = bl[i];
  if (blk < 0) return false;
  if (blk >= m) {
    set_error(err, 2u);
    return false;
  }
  const int t = blk * B + o;
  *tok = t;
  return t < n;
}

}  // namespace tls
