// Device-side helpers shared by the library's HIP translation units (gfx950 only).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace agrl {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Bits of the per-device error word (read and cleared by agrl_get_device_error).
enum : int {
  ERR_TOKEN_ID = 1,    // token_id of an action token outside [0, V)
  ERR_TRAJ_ID = 2,     // traj_id >= n_traj
  ERR_TASK_ID = 4,     // traj_task outside [0, n_task)
  ERR_GROUP_ID = 8,    // traj_group outside [0, n_group)
  ERR_MAX_ACT = 16,    // more action tokens than the workspace was laid out for
};

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
  return __uint_as_float((uint32_t)b << 16);
}

// fp32 -> bf16 bits, round to nearest even (NaN kept quiet).
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ void set_error(int* err, int bit) {
  if (err) atomicOr(err, bit);
}

template <typename T>
__host__ __device__ __forceinline__ T cdiv(T a, T b) {
  return (a + b - 1) / b;
}

}  // namespace agrl

// Host-side helpers implemented in abi.cpp.
extern "C++" {
namespace agrl {
int* device_error_ptr();          // this device's error word (nullptr on failure)
int device_cu_count();            // compute units of the current device
int hip_status(hipError_t e);     // AGRL_OK or AGRL_E_HIP, records the message
void set_last_error(const char* msg);
}  // namespace agrl
}
