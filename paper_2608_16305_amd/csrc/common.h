// Shared device/host helpers for the mtgnn HIP library (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_bf16.h>
#include <stdint.h>
#include <stddef.h>

#include "mtgnn.h"

namespace mtgnn {

// ------------------------------------------------------------------ status plumbing

// Records the HIP error string of the most recent failed launch (per thread).
void set_hip_error(hipError_t e, const char* where);

#define MTGNN_CHECK_LAUNCH(where)                                  \
  do {                                                             \
    hipError_t _e = hipGetLastError();                             \
    if (_e != hipSuccess) {                                        \
      ::mtgnn::set_hip_error(_e, where);                           \
      return MTGNN_EHIP;                                           \
    }                                                              \
  } while (0)

#define MTGNN_TRY(expr)                                            \
  do {                                                             \
    mtgnn_status _s = (expr);                                      \
    if (_s != MTGNN_OK) return _s;                                 \
  } while (0)

// ------------------------------------------------------------------ launch timer (instrumentation)

// When armed through mtgnn_timer_start(name, n), the next n launches whose
// timer name equals `name` are bracketed by HIP events on their stream.
extern bool g_timer_armed;
bool timer_begin(const char* name, hipStream_t s);
void timer_end(hipStream_t s);

struct TimedScope {
  bool on = false;
  hipStream_t s;
  TimedScope(const char* name, hipStream_t st) : s(st) {
    if (g_timer_armed) on = timer_begin(name, s);
  }
  ~TimedScope() {
    if (on) timer_end(s);
  }
};

// ------------------------------------------------------------------ small helpers

constexpr int WAVE = 64;

__host__ __device__ inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Effective count: the host-side maximum clamped by an optional device-side count.
__device__ inline int64_t eff_count(int64_t host_max, const int32_t* dev_count) {
  if (dev_count == nullptr) return host_max;
  int64_t c = (int64_t)(*dev_count);
  return c < host_max ? c : host_max;
}

// bf16 <-> fp32.  Storage conversion rounds to nearest even.
__device__ __forceinline__ float bf16_to_f32(uint16_t v) {
  return __uint_as_float(((uint32_t)v) << 16);
}
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);   // quiet NaN
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
  __device__ __forceinline__ static float load(const float* p, int64_t i) { return p[i]; }
  __device__ __forceinline__ static void store(float* p, int64_t i, float v) { p[i] = v; }
};
template <> struct Elem<uint16_t> {   // bf16 bit patterns
  __device__ __forceinline__ static float load(const uint16_t* p, int64_t i) { return bf16_to_f32(p[i]); }
  __device__ __forceinline__ static void store(uint16_t* p, int64_t i, float v) { p[i] = f32_to_bf16(v); }
};

// Cosine time encoding argument w*dt + b, rounded after the product and again
// after the sum (no fused multiply-add), so every caller rounds it identically.
__device__ __forceinline__ float time_arg(float w, float dt, float b) {
#pragma clang fp contract(off)
  float p = w * dt;
  float a = p + b;
  return a;
}

// cos(arg) as it enters a bfloat16 matrix input.  The rounding to bfloat16 (nearest, ties to even)
// is a quantisation: it must be decided on the correctly rounded float32 cosine, not on a float32
// routine's approximation of it, or a value that lies near a bfloat16 rounding midpoint can round
// the other way.  The float32 cosine is within a few units in the last place; when its 16 discarded
// bits lie within 16 units of the midpoint 0x8000, the cosine is recomputed in double precision and
// rounded to float32, which is then the correctly rounded value except within 2^-29 relative of a
// float32 midpoint.
__device__ __forceinline__ float cos_for_bf16(float arg) {
  float y = cosf(arg);
  const int low = (int)(__float_as_uint(y) & 0xFFFFu) - 0x8000;
  if (low >= -16 && low <= 16) y = (float)cos((double)arg);
  return y;
}

// Keeps a loaded 32-bit value in its register whatever the lanes do next.  A load whose result is used
// only under a per-lane condition may be moved into that condition's branch, where it is waited for on
// the spot; issuing a batch of loads, then this on each, keeps them all in flight together.
template <class T>
__device__ __forceinline__ void keep_live(T& v) {
  static_assert(sizeof(T) == 4, "one 32-bit register");
  asm volatile("" : "+v"(v));
}

__device__ __forceinline__ float sigmoidf_(float x) { return 1.0f / (1.0f + expf(-x)); }
// Gate nonlinearities on the hardware base-2 exponential and reciprocal (about 1 ulp each):
// sigma(x) = 1 / (1 + 2^(-x log2 e)),  tanh(x) = 1 - 2 / (1 + 2^(2 x log2 e)).  Both saturate correctly
// (2^(+large) = inf, 1 / inf = 0); tanh's absolute error stays near 1e-7 around zero.
__device__ __forceinline__ float sigmoid_hw(float x) {
  return __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-1.4426950408889634f * x));
}
__device__ __forceinline__ float tanh_hw(float x) {
  return 1.f - 2.f * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(2.8853900817779268f * x));
}

// Wave-level reductions (wave64).
__device__ __forceinline__ float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// ------------------------------------------------------------------ library-internal primitives

// Stable LSD radix sort of (key, value) pairs on the low `bits` bits of the key.
// The passes ping-pong between the inputs and the first radix_sort_result_bytes(n)
// of the workspace; *keys / *vals are updated to the buffers holding the result
// (so that part of the workspace must stay untouched while the result is used).
size_t radix_sort_ws_bytes(int64_t n);
size_t radix_sort_result_bytes(int64_t n);
mtgnn_status radix_sort_pairs(uint32_t** keys, uint32_t** vals, int64_t n, int bits, void* ws, size_t ws_bytes,
                              hipStream_t s);
int radix_passes(int bits);
// Where radix_sort_pairs(keys, vals, n, bits, ws, ...) leaves the sorted pairs, without sorting.
void radix_sort_output(uint32_t** keys, uint32_t** vals, int64_t n, int bits, void* ws);

// Exclusive prefix sum of int32 counts; optional device total.
size_t scan_ws_bytes(int64_t n);
mtgnn_status scan_exclusive(const int32_t* in, int32_t* out, int64_t n, int32_t* total, void* ws,
                            size_t ws_bytes, hipStream_t s);

// Deterministic column sums of a row-major [rows x cols] fp32 matrix (rows clamped by rows_dev).
size_t colsum_ws_bytes(int64_t rows, int cols);
mtgnn_status colsum(const float* X, int64_t ld, int64_t rows, const int32_t* rows_dev, int cols, float* out,
                    bool accumulate, void* ws, size_t ws_bytes, hipStream_t s);

int bits_for(int64_t max_value);   // bits needed to hold values 0..max_value

// Deterministic per-row sums over occurrences sorted by row (attention.hip): D[r] (row stride dm) = the sum,
// over the sorted positions p with skeys[p] == r and in that order, of src[svals[p]] (row stride ld, dm
// columns); rows r below the device row count with no occurrence get zeros.  Keys past the rows are
// `max_rows` (they sort last).  dm <= 512.
size_t segsum_rows_ws_bytes(int64_t n_occ, int64_t max_rows, int dm);
mtgnn_status segsum_rows(const uint32_t* skeys, const uint32_t* svals, int64_t n_occ, const float* src, int64_t ld,
                         int dm, const int32_t* n_rows, int64_t max_rows, float* D, void* ws, size_t ws_bytes,
                         hipStream_t s);

}  // namespace mtgnn
