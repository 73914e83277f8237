// Declarations of the decode step, shared by hifa4_decode.hip and the ABI.
#pragma once

#include "hifa4_internal.h"

namespace hifa4 {

// One decode step over a packed HIF4 cache (one query row per sequence).
struct DecodeLaunch {
  const half_t* q;         // [batch, Hq, D] fp16
  const float* s;          // smoothing scales or nullptr
  const int* cu;           // cu_seqlens of the cached tokens or nullptr
  const uint8_t* kc;       // canonical K^ cache [tokens, Hkv, D/64, 32]
  const uint32_t* km;
  const uint8_t* vc;       // canonical V^ cache [batch, NB, Hkv, D, 32]
  const uint32_t* vm;
  half_t* o;               // [batch, Hq, D]
  float* lse;              // [Hq, batch]
  uint8_t* dbg_codes;      // optional P^ dump [Hq, batch, NB, 32]
  uint32_t* dbg_meta;
  uint8_t* ws;
  hipEvent_t* ev;          // optional; ev[1] is recorded before the merge kernel
  int batch, S, NB, hq, hkv, D, norm;
  int test_no_publish;     // testing: no run maxima published, waits give up after 16 polls
  float c;
};

size_t decode_workspace_bytes(int batch, int hq, int hkv, int D, int NB);
hipError_t launch_decode(const DecodeLaunch& d, hipStream_t st);

}  // namespace hifa4
