// Durations generated on the device: a strategy-knob grid of base durations
// times a per-(op, scenario) noise factor from a counter-based generator.
// Replaces the duration matrix when the scenarios are a sweep over knobs with
// profiling noise (the paper's motivation: many parallelisation strategies
// and configurations evaluated by simulation, Sec. 1; profiled op times vary
// by under 1 % of their mean, Sec. 3).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mlsim {

// Generation parameters of one call (kernel argument; every field uniform).
struct DurGen {
  const int32_t *base;  // device [n_knobs][n_ops]: base ns of op v under knob k at k * n_ops + v
  int32_t n_ops;
  int32_t n_knobs;
  int64_t knob_block;   // consecutive global scenarios sharing a knob
  int64_t scen0;        // global index of scenario 0 of the call
  uint32_t noise;       // noise multiplier, < 2^20
  uint32_t key0, key1;  // Philox key: low and high words of the seed
};

constexpr int32_t kGenBaseMax = 1 << 24;  // largest valid base (ns)
constexpr uint32_t kGenNoiseMax = 1u << 20;

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds, each taking
// the two 32x32 -> 64-bit products of words 0 and 2 with the round
// multipliers and producing (hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0), the key
// advancing by the Weyl constants after every round.  The key is
// wave-uniform, so its schedule stays in scalar registers.
__device__ __forceinline__ void philox4x32_10(uint32_t &x0, uint32_t &x1, uint32_t &x2, uint32_t &x3,
                                              uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * x0;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * x2;
    const uint32_t y0 = (uint32_t)(p1 >> 32) ^ x1 ^ k0;
    const uint32_t y2 = (uint32_t)(p0 >> 32) ^ x3 ^ k1;
    x1 = (uint32_t)p1;
    x3 = (uint32_t)p0;
    x0 = y0;
    x2 = y2;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
}

// Duration of op v in global scenario S = (s_hi, s_lo) with base b:
//   (x0..x3) = Philox4x32-10((s_lo, s_hi, v, 0), (key0, key1)),
//   U = sum of the eight 16-bit halves of x0..x3 (Irwin-Hall of 8 uniforms),
//   t = 2U - 524280 (zero mean), d = b + floor((b t noise + 2^39) / 2^40),
// exact in 64-bit integers (|b t noise| < 2^24 2^19 2^20 = 2^63).  A base
// outside [1, 2^24] gives 0, which the replay reports as a bad duration.
// With noise < 2^20 the adjustment stays below b / 2, so d >= 1.
__device__ __forceinline__ int32_t gen_duration(int32_t b, uint32_t s_lo, uint32_t s_hi, uint32_t v,
                                                uint32_t k0, uint32_t k1, uint32_t noise) {
  uint32_t x0 = s_lo, x1 = s_hi, x2 = v, x3 = 0;
  philox4x32_10(x0, x1, x2, x3, k0, k1);
  const uint32_t u = (x0 & 0xFFFFu) + (x0 >> 16) + (x1 & 0xFFFFu) + (x1 >> 16) + (x2 & 0xFFFFu) +
                     (x2 >> 16) + (x3 & 0xFFFFu) + (x3 >> 16);
  const int32_t t = 2 * (int32_t)u - 524280;
  const bool ok = (uint32_t)(b - 1) < (uint32_t)kGenBaseMax;
  const int32_t bb = ok ? b : 0;
  const int64_t q = (int64_t)bb * t * (int64_t)noise;
  const int32_t adj = (int32_t)((q + (1ll << 39)) >> 40);
  return ok ? bb + adj : 0;
}

// Row of base durations for the knob of global scenario S.
__device__ __forceinline__ const int32_t *gen_knob_row(const DurGen &g, int64_t S) {
  const int64_t k = (S / g.knob_block) % g.n_knobs;
  return g.base + k * (int64_t)g.n_ops;
}

}  // namespace mlsim
