// Device helpers shared by the HIP sources of libeta (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "eta_internal.h"

namespace eta {

constexpr float kNegInf = -__builtin_inff();

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// two fp32 -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// a sequence length clamped to [0, cap]
__device__ __forceinline__ int64_t clamp_len(const int32_t* seq_lens, int b, int64_t cap) {
  int64_t T = seq_lens[b];
  return T < 0 ? 0 : (T > cap ? cap : T);
}

// Launch wrapped by the optional per-kernel hook (timing / tracing); returns
// the launch error.
template <typename F>
hipError_t with_hook(LaunchHook hook, int kind, hipStream_t st, F&& f) {
  if (hook) hook(kind, st, false);
  f();
  hipError_t e = hipGetLastError();
  if (hook) hook(kind, st, true);
  return e;
}

}  // namespace eta
