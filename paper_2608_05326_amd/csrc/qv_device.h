// Device-side helpers shared by the gfx950 kernels: vector types, exact
// fp16 / bf16 conversions and the launch argument blocks.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qv_layout.h"

namespace qv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

struct AttnArgs {
  Geometry g;
  UnitLayout L;
  uint8_t* base;            // unit block of (layer, seq 0)
  const uint16_t* q;        // [B][H_q][d]
  const uint16_t* k_new;    // [B][H_kv][d]
  const uint16_t* v_new;
  void* out;                // [B][H_q][d]
  int32_t T;                // sequence length after appending this step's token
  int32_t ring_w0;          // first window not routed yet
  int32_t n_ring;           // windows in [ring_w0, ring_w0 + n_ring) are attended from the ring
  int32_t n_sink_items;     // sink slots holding sink tokens
  float decay;              // factor on every updated window score before this step's mass
  int32_t key_norm;         // 1: key-norm scores (no attention masses; the new token's key norm)
  float pnorm_p;            // > 0: attention p-norm scores with this p
  int32_t period_start;     // 1: first step after a routing event (or prefill)
};

// Routing events of up to kRouteBatch layers go to one launch (one workgroup row
// per layer): the per-layer part of an event.
constexpr int kRouteBatch = 8;
// polls of the routing stream's wait for the cache stream before it gives up even
// if the wall clock has not passed its limit (each poll sleeps about 1024 clocks)
constexpr int64_t kGateMaxPolls = 40000000;
struct RetierUnit {
  uint8_t* base;            // the layer's first unit (sequence 0)
  int32_t aged_w0, aged_w1; // aged windows entering the candidate pool
  // split plans for the decode steps up to the next routing event, one per slot:
  // the sequence lengths [plan_t0, plan_t1] it serves (plan_t0 <= 0: none) and the
  // recent-region + sink windows those steps attend after the live list
  int32_t plan_t0[kPlanSlots], plan_t1[kPlanSlots];
  int32_t plan_extra[kPlanSlots];
};

struct RetierArgs {
  Geometry g;
  UnitLayout L;
  int32_t prefill;          // 1: candidates are the prompt's historical windows
  const float* init_scores; // prefill: [B][n_init]
  int32_t n_init;
  int32_t n_units;          // layers of this launch: workgroup row y serves unit[y]
  RetierUnit unit[kRouteBatch];
  const int32_t* gate_fail; // routing stream: nonzero when its wait for the cache stream timed out
};

struct MigrateArgs {
  Geometry g;
  UnitLayout L;
  int32_t n_units;          // layers of this launch: workgroup layer z serves base[z]
  uint8_t* base[kRouteBatch];
  const uint16_t* src_k;    // prompt keys [B][H_kv][T][d] (prefill only)
  const uint16_t* src_v;
  int32_t src_T;
  const int32_t* gate_fail; // as RetierArgs::gate_fail
};

struct KeyNormArgs {        // key-norm scores of the prompt windows
  Geometry g;
  const uint16_t* k;        // [B][H_kv][T][d] bf16 prompt keys
  int32_t T, n_init;
  float* out;               // [B][n_init]
};

// max / sum over the four 16-lane rows: lanes i, i^16, i^32, i^48 (gfx950 permlane
// swaps; every lane of the four gets the same value)
__device__ __forceinline__ float rows_max(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const uint32_t a0 = a[0], a1 = a[1];
  const float y = fmaxf(__uint_as_float(a0), __uint_as_float(a1));
  const uint32_t v = __float_as_uint(y);
  const auto b = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  const uint32_t b0 = b[0], b1 = b[1];
  return fmaxf(__uint_as_float(b0), __uint_as_float(b1));
}
__device__ __forceinline__ float rows_sum(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const uint32_t a0 = a[0], a1 = a[1];
  const float y = __uint_as_float(a0) + __uint_as_float(a1);
  const uint32_t v = __float_as_uint(y);
  const auto b = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  const uint32_t b0 = b[0], b1 = b[1];
  return __uint_as_float(b0) + __uint_as_float(b1);
}

struct ObsArgs {            // initial window scores from the observation queries' attention
  const uint16_t* q;        // [B][H_q][n_obs][d] bf16
  const uint16_t* k;        // [B][H_kv][T][d] bf16
  int32_t B, H_q, H_kv, gqa, T, n_obs, n_rows, W, sink, n_w;
  int32_t cbase;            // first key of chunk 0 (sink - 64 n_pre, <= 0)
  int32_t n_pre;            // chunks before the first window (sink keys)
  int32_t n_chunks;         // chunks of 64 keys
  int32_t n_blk;            // workgroups of four chunks
  float scale_log2;
  float2* cml;              // [B][H_kv][n_chunks][n_rows] (max, exp-sum) per chunk and row
  float* wl;                // [B][H_kv][n_w][n_rows] window exp-sum relative to its chunk's max
  float2* row_ml;           // [B][H_kv][n_rows] (M, 1 / L)
  float* scores;            // [B][n_w]
};

struct ScorePowArgs {       // p-norm ranking: prompt scores raised to the power p
  const float* in;
  float* out;
  int32_t n;
  float p;
};

struct PackArgs {           // copy prompt tokens into ring / sink slots
  Geometry g;
  UnitLayout L;
  uint8_t* base;
  const uint16_t* src_k;
  const uint16_t* src_v;
  int32_t src_T;
  int32_t tok0, tok1;       // token range [tok0, tok1) to copy
};

__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

__device__ inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ inline double fp16_bits_to_f64(uint16_t h) {
  return (double)(float)__builtin_bit_cast(_Float16, h);
}

// next fp16 value toward -inf / +inf (finite inputs)
__device__ inline uint16_t fp16_next_down(uint16_t h) {
  if ((h & 0x7FFFu) == 0) return 0x8001u;
  return (h & 0x8000u) ? (uint16_t)(h + 1) : (uint16_t)(h - 1);
}
__device__ inline uint16_t fp16_next_up(uint16_t h) {
  if ((h & 0x7FFFu) == 0) return 0x0001u;
  return (h & 0x8000u) ? (uint16_t)(h - 1) : (uint16_t)(h + 1);
}

// largest fp16 <= x (x finite, |x| <= 65504)
__device__ inline uint16_t fp16_round_down(float x) {
  uint16_t h = __builtin_bit_cast(uint16_t, (_Float16)x);
  if ((float)__builtin_bit_cast(_Float16, h) > x) h = fp16_next_down(h);
  return h;
}

// exact float64 -> bf16, round to nearest even, single rounding
__device__ inline uint16_t f64_to_bf16_rne(double x) {
  uint64_t u = __double_as_longlong(x);
  uint16_t sign = (uint16_t)((u >> 48) & 0x8000u);
  uint64_t a = u & 0x7FFFFFFFFFFFFFFFull;
  if (a == 0) return sign;
  int e = (int)(a >> 52) - 1023;
  if (e >= -126) {
    uint64_t mant = a & ((1ull << 52) - 1);
    uint64_t m7 = mant >> 45, rem = mant & ((1ull << 45) - 1), half = 1ull << 44;
    if (rem > half || (rem == half && (m7 & 1))) m7 += 1;
    if (m7 == 128) { m7 = 0; e += 1; }
    if (e > 127) return (uint16_t)(sign | 0x7F80u);
    return (uint16_t)(sign | ((uint32_t)(e + 127) << 7) | (uint32_t)m7);
  }
  // below the bf16 normal range: integer multiple of 2^-133
  double y = __builtin_rint(__builtin_fabs(x) * 0x1p133);
  return (uint16_t)(sign | (uint16_t)y);
}

__device__ inline void set_error(int32_t* counts, int32_t bits) {
  __hip_atomic_fetch_or(counts + CNT_ERROR, bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace qv
