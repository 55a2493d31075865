// Internal helpers shared by the libseg translation units (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <string>

#include "seg.h"

namespace seg {

// ---------------------------------------------------------------- errors
void set_error(const std::string &msg);
void clear_error();

struct Fail {
  seg_status status;
};

#define SEG_CHECK(cond, code, ...)                                   \
  do {                                                               \
    if (!(cond)) {                                                   \
      char _b[512];                                                  \
      snprintf(_b, sizeof(_b), __VA_ARGS__);                         \
      ::seg::set_error(_b);                                          \
      throw ::seg::Fail{code};                                       \
    }                                                                \
  } while (0)

#define SEG_HIP(expr)                                                          \
  do {                                                                         \
    hipError_t _e = (expr);                                                    \
    if (_e != hipSuccess) {                                                    \
      ::seg::set_error(std::string(#expr) + ": " + hipGetErrorString(_e));     \
      throw ::seg::Fail{SEG_ERR_HIP};                                          \
    }                                                                          \
  } while (0)

#define SEG_LAUNCH_CHECK() SEG_HIP(hipGetLastError())

// Run `body` and turn failures into a status (no exception crosses the ABI).
template <class F>
inline seg_status guarded(F &&body) {
  try {
    clear_error();
    body();
    return SEG_OK;
  } catch (const Fail &f) {
    return f.status;
  } catch (const std::exception &e) {
    set_error(std::string("internal error: ") + e.what());
    return SEG_ERR_ARG;
  } catch (...) {
    set_error("internal error");
    return SEG_ERR_ARG;
  }
}

// Brackets one kernel launch with HIP events when timing is enabled
// (seg_profile_enable); a no-op otherwise.
class ProfScope {
 public:
  ProfScope(const char *name, hipStream_t s);
  ~ProfScope();
  ProfScope(const ProfScope &) = delete;
  ProfScope &operator=(const ProfScope &) = delete;

 private:
  const char *name_;
  hipStream_t stream_;
  hipEvent_t start_{}, stop_{};
  bool active_ = false;
};

inline size_t align_up(size_t x, size_t a = 256) { return (x + a - 1) / a * a; }

// Carves aligned sub-buffers out of a caller workspace.
struct Carver {
  char *base;
  size_t off = 0;
  explicit Carver(void *b) : base(static_cast<char *>(b)) {}
  template <class T>
  T *take(size_t count) {
    T *p = reinterpret_cast<T *>(base ? base + off : nullptr);
    off = align_up(off + count * sizeof(T));
    return p;
  }
};

// ---------------------------------------------------------------- device
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ unsigned short f2bf_bits(float x) {
  __bf16 b = (__bf16)x;  // round to nearest even
  return __builtin_bit_cast(unsigned short, b);
}
__device__ __forceinline__ float bf_bits2f(unsigned short b) {
  return __builtin_bit_cast(float, (unsigned)b << 16);
}

// Load a value of the kernel input dtype and round it to bf16 bits.
template <class T>
__device__ __forceinline__ unsigned short load_bf(const T *p, long i);
template <>
__device__ __forceinline__ unsigned short load_bf<unsigned short>(const unsigned short *p, long i) {
  return p[i];
}
template <>
__device__ __forceinline__ unsigned short load_bf<float>(const float *p, long i) {
  return f2bf_bits(p[i]);
}

template <class T>
__device__ __forceinline__ void store_val(T *p, long i, float v);
template <>
__device__ __forceinline__ void store_val<unsigned short>(unsigned short *p, long i, float v) {
  p[i] = f2bf_bits(v);
}
template <>
__device__ __forceinline__ void store_val<float>(float *p, long i, float v) {
  p[i] = v;
}

__device__ __forceinline__ f32x16 mfma32(const bf16x8 &a, const bf16x8 &b, const f32x16 &c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Position p (0..15) inside a 16-element chunk of a transposed tile holds the
// element of offset kperm(p) of that chunk.  It matches the order in which the
// 32x32 MFMA accumulator of a lane holds its rows: lane half h, register j of a
// 16-row chunk holds row 8*(j/4) + 4*h + j%4, and an operand lane half h reads
// positions 8h..8h+7.  The map is an involution (it swaps 4..7 with 8..11).
__host__ __device__ __forceinline__ int kperm(int p) {
  return (p & ~12) | ((p & 4) << 1) | ((p & 8) >> 1);
}

// dst[i] = value for i < n 32-bit words.  Compute entry points clear their
// outputs with this kernel rather than hipMemsetAsync, so a caller can
// capture them in a HIP graph and replay it.
namespace {
__global__ void __launch_bounds__(256) k_fill32(uint32_t *__restrict__ dst, long n, uint32_t value) {
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x)
    dst[i] = value;
}
}  // namespace

inline void fill32(void *dst, long n, uint32_t value, hipStream_t st) {
  if (n <= 0) return;
  const long blocks = (n + 255) / 256;
  k_fill32<<<(unsigned)(blocks < 16384 ? blocks : 16384), 256, 0, st>>>(static_cast<uint32_t *>(dst), n,
                                                                        value);
  SEG_LAUNCH_CHECK();
}

}  // namespace seg
