// Task advantage normalisation (AgentRL Sec. 3.2) on top of GRPO's group-relative
// advantage (App. B.2), for a global batch of trajectories.
//
// Compiled with -ffp-contract=off: every + - * / and sqrtf below is one correctly
// rounded fp32 operation, so the results are bit-identical to any implementation
// that follows the same summation order (see agrl.h).
#include <math.h>

#include "../../include/agrl.h"
#include "common.hpp"

namespace agrl {
namespace {

constexpr int kCountPerLane = 16;

__global__ void fill_i32_kernel(int32_t* p, int64_t n, int32_t v) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// n_tau: each lane walks kCountPerLane consecutive tokens, adding runs of the
// same trajectory; the wave then merges lanes that end on the same trajectory.
// Integer atomics are exact, so the counts do not depend on the order.
// VEC: traj_id and mask are 16-byte aligned, and a lane's whole run of tokens
// is read with four 16-byte id loads and one 16-byte mask load.
template <bool VEC>
__global__ __launch_bounds__(256) void count_kernel(int64_t T_g, int32_t n_traj,
                                                    const int32_t* __restrict__ traj_id,
                                                    const uint8_t* __restrict__ mask,
                                                    int32_t* act_count, int* err) {
  static_assert(kCountPerLane == 16, "one 16-byte mask load per lane");
  const int64_t t0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * kCountPerLane;
  int cur = -1, cnt = 0;
  auto token = [&](int id, bool m) {
    if (id >= n_traj) {
      set_error(err, ERR_TRAJ_ID);
      return;
    }
    if (id < 0 || !m) return;
    if (id != cur) {
      if (cnt) atomicAdd(&act_count[cur], cnt);
      cur = id;
      cnt = 0;
    }
    ++cnt;
  };
  if (VEC && t0 + kCountPerLane <= T_g) {
    typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
    i32x4 ids[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) ids[k] = *(const i32x4*)(traj_id + t0 + 4 * k);
    const u32x4 mw = *(const u32x4*)(mask + t0);
#pragma unroll
    for (int i = 0; i < kCountPerLane; ++i)
      token(ids[i >> 2][i & 3], (mw[i >> 2] >> (8 * (i & 3))) & 0xFFu);
  } else {
    for (int i = 0; i < kCountPerLane; ++i) {
      const int64_t t = t0 + i;
      if (t >= T_g) break;
      token(traj_id[t], mask[t] != 0);
    }
  }
  const int lane = threadIdx.x & 63;
  for (;;) {
    const uint64_t pend = __ballot(cnt > 0);
    if (!pend) break;
    const int leader = __ffsll((unsigned long long)pend) - 1;
    const int lid = __shfl(cur, leader);
    int mine = (cnt > 0 && cur == lid) ? cnt : 0;
    for (int o = 32; o >= 1; o >>= 1) mine += __shfl_xor(mine, o);
    if (lane == leader) atomicAdd(&act_count[lid], mine);
    if (cnt > 0 && cur == lid) cnt = 0;
  }
}

// Lowest and highest trajectory index per segment key, one atomic pair per
// distinct key of the wave: the wave's trajectories are consecutive, so the
// lowest lane holding a key has its lowest index and the highest lane its highest.
__device__ __forceinline__ void wave_range(bool valid, int key, int tau, int32_t* range) {
  const int lane = threadIdx.x & 63;
  uint64_t pend = __ballot(valid);
  while (pend) {
    const int k = __shfl(key, __ffsll((unsigned long long)pend) - 1);
    const uint64_t m = __ballot(valid && key == k);
    if (lane == __ffsll((unsigned long long)m) - 1) atomicMin(&range[2 * k], tau);
    if (lane == 63 - __clzll((unsigned long long)m)) atomicMax(&range[2 * k + 1], tau);
    pend &= ~m;
  }
}

// Zero the per-trajectory counts and check the task / group ids, one launch.
// With `range` (2 ints per group, then 2 per task, preset to (n_traj, -1)),
// also record the lowest and the highest index of each group's and each
// task's members (integer atomics: the result does not depend on the order).
__global__ void prep_kernel(int32_t n_traj, int32_t n_task, int32_t n_group,
                            const int32_t* traj_task, const int32_t* traj_group,
                            int32_t* act_count, int32_t* range, int* err) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  const bool in = j < n_traj;
  const int i = in ? traj_task[j] : 0;
  const int g = in && traj_group ? traj_group[j] : 0;
  const bool ok_task = in && i >= 0 && i < n_task;
  const bool ok_group = in && traj_group && g >= 0 && g < n_group;
  if (in) {
    act_count[j] = 0;
    if (!ok_task) set_error(err, ERR_TASK_ID);
    if (traj_group && !ok_group) set_error(err, ERR_GROUP_ID);
  }
  if (range) {
    if (traj_group) wave_range(ok_group, g, j, range);
    wave_range(ok_task, i, j, range + 2 * n_group);
  }
}

// Preset the member ranges to empty: lowest = n_traj, highest = -1.
__global__ void range_init_kernel(int32_t n, int32_t n_traj, int32_t* range) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k < n) range[k] = (k & 1) ? -1 : n_traj;
}

// The trajectories a segment's wave visits: [first, last] of its members when
// the ranges were recorded, else all of them.  The wave walks them in steps of
// 64 from first rounded down to a multiple of 64, so that lane l always takes
// the trajectories tau = l mod 64 in ascending order: the summation order, and
// so every bit of the result, is the same either way.
struct Span {
  int first, last;
};
__device__ __forceinline__ Span segment_span(const int32_t* range, int k, int32_t n_traj) {
  if (!range) return Span{0, n_traj - 1};
  return Span{range[2 * k], range[2 * k + 1]};
}

// The fixed combination of a wave's 64 partial sums: acc_l += acc_{l xor o},
// o = 32 .. 1.  All lanes end with the same bits.
__device__ __forceinline__ float butterfly_sum(float acc) {
  for (int o = 32; o >= 1; o >>= 1) acc = acc + __shfl_xor(acc, o);
  return acc;
}

__device__ __forceinline__ int64_t wave_sum_i64(int64_t v) {
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// GRPO stage: one wave per group.  Lane l owns trajectories l, l+64, ...
// With drop_uniform, a group whose rewards are all equal is marked dropped by a
// quiet NaN in a_hat (the task stage leaves such trajectories out and gives
// them advantage 0).
__device__ void group_wave(int g, int lane, int32_t n_traj, Span sp,
                           const int32_t* __restrict__ traj_group,
                           const float* __restrict__ reward, int32_t ddof, float eps,
                           int32_t drop_uniform, float* a_hat) {
  if (sp.last < sp.first) return;      // no members
  const int t0 = (sp.first & ~63) + lane, end = sp.last + 1;
  float acc = 0.0f;
  int K = 0;
  for (int base = sp.first & ~63; base < end; base += 64) {
    const int tau = base + lane;
    const bool mem = tau < end && traj_group[tau] == g;
    if (mem) acc = acc + reward[tau];
    K += __popcll(__ballot(mem));
  }
  if (K == 0) return;
  if (drop_uniform) {
    // exact: min and max over the members do not depend on the order
    float lo = INFINITY, hi = -INFINITY;
    for (int tau = t0; tau < end; tau += 64)
      if (traj_group[tau] == g) {
        lo = fminf(lo, reward[tau]);
        hi = fmaxf(hi, reward[tau]);
      }
    for (int o = 32; o >= 1; o >>= 1) {
      lo = fminf(lo, __shfl_xor(lo, o));
      hi = fmaxf(hi, __shfl_xor(hi, o));
    }
    if (lo == hi) {
      for (int tau = t0; tau < end; tau += 64)
        if (traj_group[tau] == g) a_hat[tau] = __builtin_nanf("");
      return;
    }
  }
  if (K - ddof <= 0) {
    for (int tau = t0; tau < end; tau += 64)
      if (traj_group[tau] == g) a_hat[tau] = 0.0f;
    return;
  }
  const float mu = butterfly_sum(acc) / (float)K;
  acc = 0.0f;
  for (int tau = t0; tau < end; tau += 64) {
    if (traj_group[tau] == g) {
      const float dv = reward[tau] - mu;
      acc = acc + dv * dv;
    }
  }
  const float var = butterfly_sum(acc) / (float)(K - ddof);
  const float den = sqrtf(var) + eps;
  for (int tau = t0; tau < end; tau += 64)
    if (traj_group[tau] == g) a_hat[tau] = (reward[tau] - mu) / den;
}

__global__ __launch_bounds__(256) void group_kernel(int32_t n_group, int32_t n_traj,
                                                    const int32_t* __restrict__ traj_group,
                                                    const float* __restrict__ reward,
                                                    const int32_t* range, int32_t ddof, float eps,
                                                    int32_t drop_uniform, float* a_hat) {
  const int g = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (g < n_group)
    group_wave(g, threadIdx.x & 63, n_traj, segment_span(range, g, n_traj), traj_group, reward,
               ddof, eps, drop_uniform, a_hat);
}

// Task stage: one wave per task; statistics of the token-level set, where
// trajectory tau contributes its advantage with multiplicity n_tau.
// src may alias adv_traj: each lane reads its own trajectories before writing them.
// With drop_uniform, trajectories whose group stage left a NaN mark (dropped
// groups) are not members of their task's set and get advantage 0.
__device__ void task_wave(int i, int lane, int32_t n_traj, Span sp,
                          const int32_t* __restrict__ traj_task,
                          const int32_t* __restrict__ act_count, const float* src, int32_t ddof,
                          float eps, int32_t drop_uniform, int64_t* task_count, float* task_mean,
                          float* task_std, float* adv_traj) {
  auto member = [&](int tau) {
    return traj_task[tau] == i && !(drop_uniform && isnan(src[tau]));
  };
  const int t0 = (sp.first & ~63) + lane, end = sp.last + 1;   // empty when last < first
  float acc = 0.0f;
  int64_t n_lane = 0;
  for (int tau = t0; tau < end; tau += 64) {
    if (member(tau)) {
      const int n = act_count[tau];
      n_lane += n;
      acc = acc + (float)n * src[tau];
    }
  }
  const int64_t N = wave_sum_i64(n_lane);
  if (N == 0) {
    for (int tau = t0; tau < end; tau += 64)
      if (traj_task[tau] == i) adv_traj[tau] = 0.0f;       // dropped ones included
    if (lane == 0) {
      task_count[i] = 0;
      task_mean[i] = 0.0f;
      task_std[i] = 0.0f;
    }
    return;
  }
  const float mu = butterfly_sum(acc) / (float)N;
  acc = 0.0f;
  for (int tau = t0; tau < end; tau += 64) {
    if (member(tau)) {
      const float dv = src[tau] - mu;
      acc = acc + (float)act_count[tau] * (dv * dv);
    }
  }
  const float q = butterfly_sum(acc);
  const float sigma = (N - ddof > 0) ? sqrtf(q / (float)(N - ddof)) : 0.0f;
  const float den = sigma + eps;
  for (int tau = t0; tau < end; tau += 64)
    if (traj_task[tau] == i) adv_traj[tau] = member(tau) ? (src[tau] - mu) / den : 0.0f;
  if (lane == 0) {
    task_count[i] = N;
    task_mean[i] = mu;
    task_std[i] = sigma;
  }
}

__global__ __launch_bounds__(256) void task_kernel(int32_t n_task, int32_t n_group, int32_t n_traj,
                                                   const int32_t* __restrict__ traj_task,
                                                   const int32_t* __restrict__ act_count,
                                                   const float* src, const int32_t* range,
                                                   int32_t ddof, float eps, int32_t drop_uniform,
                                                   int64_t* task_count, float* task_mean,
                                                   float* task_std, float* adv_traj) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i < n_task)
    task_wave(i, threadIdx.x & 63, n_traj, segment_span(range, n_group + i, n_traj),
              traj_task, act_count, src, ddof, eps, drop_uniform, task_count, task_mean,
              task_std, adv_traj);
}

// VEC: traj_id, mask and adv_tok are 16-byte aligned and a thread handles 4
// tokens with one 16-byte id load, one 4-byte mask load and one 16-byte store.
template <bool VEC>
__global__ void broadcast_kernel(int64_t T_g, int32_t n_traj, const int32_t* __restrict__ traj_id,
                                 const uint8_t* __restrict__ mask,
                                 const float* __restrict__ adv_traj, float* adv_tok) {
  auto one = [&](int id, bool m) { return (m && id >= 0 && id < n_traj) ? adv_traj[id] : 0.0f; };
  const int64_t t = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * (VEC ? 4 : 1);
  if (VEC && t + 4 <= T_g) {
    typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
    const i32x4 id = *(const i32x4*)(traj_id + t);
    const uint32_t m = *(const uint32_t*)(mask + t);
    *(f32x4*)(adv_tok + t) = f32x4{one(id[0], m & 0xFFu), one(id[1], (m >> 8) & 0xFFu),
                                   one(id[2], (m >> 16) & 0xFFu), one(id[3], m >> 24)};
    return;
  }
  for (int64_t u = t; u < T_g && u < t + (VEC ? 4 : 1); ++u) adv_tok[u] = one(traj_id[u], mask[u] != 0);
}

int fail(int code, const char* msg) {
  set_last_error(msg);
  return code;
}

// Sequence-level weights: every block counts the non-empty trajectories
// (n_traj is small) and then weighs its tokens.
__global__ __launch_bounds__(256) void seq_weight_kernel(int64_t T, int32_t n_traj,
                                                         const int32_t* __restrict__ traj_id,
                                                         const uint8_t* __restrict__ mask,
                                                         const int32_t* __restrict__ seq_count,
                                                         float* __restrict__ w) {
  __shared__ int part[256 / 64];
  int n = 0;
  for (int j = threadIdx.x; j < n_traj; j += blockDim.x) n += seq_count[j] > 0;
  for (int o = 32; o >= 1; o >>= 1) n += __shfl_xor(n, o);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = n;
  __syncthreads();
  const int n_seq = part[0] + part[1] + part[2] + part[3];
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < T;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int id = traj_id[t];
    float v = 0.0f;
    if (id >= 0 && id < n_traj && mask[t])
      v = (float)(1.0 / ((double)n_seq * (double)seq_count[id]));
    w[t] = v;
  }
}

}  // namespace
}  // namespace agrl

extern "C" int agrl_task_adv_norm(int64_t T_g, int32_t n_traj, int32_t n_task, int32_t n_group,
                                  const int32_t* traj_id, const uint8_t* action_mask,
                                  const int32_t* traj_task, const int32_t* traj_group,
                                  const float* reward, const agrl_options* opt,
                                  int32_t* act_count, int64_t* task_count, float* task_mean,
                                  float* task_std, float* adv_traj, float* adv_tok,
                                  void* stream) {
  using namespace agrl;
  if (T_g < 0 || n_traj < 0 || n_task < 0 || n_group < 0)
    return fail(AGRL_E_SHAPE, "agrl_task_adv_norm: negative size");
  if (T_g > ((int64_t)1 << 40)) return fail(AGRL_E_SHAPE, "agrl_task_adv_norm: T_g too large");
  if (traj_group && n_traj > 0 && n_group == 0)
    return fail(AGRL_E_SHAPE, "agrl_task_adv_norm: traj_group given with n_group == 0");
  if (T_g > 0 && (!traj_id || !action_mask))
    return fail(AGRL_E_NULL, "agrl_task_adv_norm: traj_id/action_mask is NULL");
  if (n_traj > 0 && (!traj_task || !reward || !act_count || !adv_traj))
    return fail(AGRL_E_NULL, "agrl_task_adv_norm: per-trajectory array is NULL");
  if (n_task > 0 && (!task_count || !task_mean || !task_std))
    return fail(AGRL_E_NULL, "agrl_task_adv_norm: per-task output is NULL");
  agrl_options o = {};
  if (opt) o = *opt;
  if (o.std_ddof != 0 && o.std_ddof != 1)
    return fail(AGRL_E_FLAGS, "agrl_task_adv_norm: std_ddof must be 0 or 1");
  if (!(o.std_eps >= 0.0f) || !isfinite(o.std_eps))
    return fail(AGRL_E_FLAGS, "agrl_task_adv_norm: std_eps must be finite and >= 0");
  const float eps = o.std_eps == 0.0f ? 1e-6f : o.std_eps;
  if (o.drop_uniform_groups != 0 && o.drop_uniform_groups != 1)
    return fail(AGRL_E_FLAGS, "agrl_task_adv_norm: drop_uniform_groups must be 0 or 1");
  if (o.drop_uniform_groups && !traj_group && n_traj > 0)
    return fail(AGRL_E_FLAGS, "agrl_task_adv_norm: drop_uniform_groups needs traj_group");

  hipStream_t s = (hipStream_t)stream;
  int* err = device_error_ptr();
  if (!err) return hip_status(hipErrorInvalidSymbol);

  // member ranges (optional scratch): groups first, then tasks
  const int32_t n_group_used = traj_group ? n_group : 0;
  int32_t* range = n_traj > 0 ? o.adv_ranges : nullptr;
  if (range && n_group_used + n_task > 0)
    hipLaunchKernelGGL(range_init_kernel, dim3(cdiv(2 * (n_group_used + n_task), 256)), dim3(256),
                       0, s, 2 * (n_group_used + n_task), n_traj, range);
  if (n_traj > 0)
    hipLaunchKernelGGL(prep_kernel, dim3(cdiv(n_traj, 256)), dim3(256), 0, s, n_traj, n_task,
                       n_group_used, traj_task, traj_group, act_count, range, err);
  const bool vec_in = (((uintptr_t)traj_id | (uintptr_t)action_mask) & 15) == 0;
  if (T_g > 0 && n_traj >= 0) {
    const int64_t lanes = cdiv<int64_t>(T_g, kCountPerLane);
    const dim3 grid((unsigned)cdiv<int64_t>(lanes, 256));
    if (vec_in)
      hipLaunchKernelGGL(count_kernel<true>, grid, dim3(256), 0, s, T_g, n_traj, traj_id,
                         action_mask, act_count, err);
    else
      hipLaunchKernelGGL(count_kernel<false>, grid, dim3(256), 0, s, T_g, n_traj, traj_id,
                         action_mask, act_count, err);
  }
  const int32_t ddof = (int32_t)o.std_ddof;
  const int32_t drop = traj_group ? o.drop_uniform_groups : 0;
  if (traj_group && n_group > 0)
    hipLaunchKernelGGL(group_kernel, dim3(cdiv(n_group, 4)), dim3(256), 0, s, n_group, n_traj,
                       traj_group, reward, (const int32_t*)range, ddof, eps, drop, adv_traj);
  if (n_task > 0)
    hipLaunchKernelGGL(task_kernel, dim3(cdiv(n_task, 4)), dim3(256), 0, s, n_task, n_group_used,
                       n_traj, traj_task, act_count,
                       traj_group ? (const float*)adv_traj : reward, (const int32_t*)range, ddof,
                       eps, drop, task_count, task_mean, task_std, adv_traj);
  if (adv_tok && T_g > 0) {
    if (vec_in && ((uintptr_t)adv_tok & 15) == 0)
      hipLaunchKernelGGL(broadcast_kernel<true>, dim3((unsigned)cdiv<int64_t>(cdiv<int64_t>(T_g, 4), 256)),
                         dim3(256), 0, s, T_g, n_traj, traj_id, action_mask,
                         (const float*)adv_traj, adv_tok);
    else
      hipLaunchKernelGGL(broadcast_kernel<false>, dim3((unsigned)cdiv<int64_t>(T_g, 256)), dim3(256),
                         0, s, T_g, n_traj, traj_id, action_mask, (const float*)adv_traj, adv_tok);
  }
  return hip_status(hipGetLastError());
}

extern "C" int agrl_sequence_mean_weights(int64_t T, int32_t n_traj, const int32_t* traj_id,
                                          const uint8_t* action_mask, int32_t* seq_count,
                                          float* token_weight, void* stream) {
  using namespace agrl;
  if (T < 0 || n_traj < 0) return fail(AGRL_E_SHAPE, "agrl_sequence_mean_weights: negative size");
  if (T > ((int64_t)1 << 40))
    return fail(AGRL_E_SHAPE, "agrl_sequence_mean_weights: T too large");
  if (T > 0 && (!traj_id || !action_mask || !token_weight))
    return fail(AGRL_E_NULL, "agrl_sequence_mean_weights: traj_id/action_mask/token_weight is NULL");
  if (n_traj > 0 && !seq_count)
    return fail(AGRL_E_NULL, "agrl_sequence_mean_weights: seq_count is NULL");
  hipStream_t s = (hipStream_t)stream;
  int* err = device_error_ptr();
  if (!err) return hip_status(hipErrorInvalidSymbol);
  if (n_traj > 0)
    hipLaunchKernelGGL(fill_i32_kernel, dim3(cdiv(n_traj, 256)), dim3(256), 0, s, seq_count,
                       (int64_t)n_traj, 0);
  if (T > 0) {
    const int64_t lanes = cdiv<int64_t>(T, kCountPerLane);
    const dim3 grid((unsigned)cdiv<int64_t>(lanes, 256));
    if ((((uintptr_t)traj_id | (uintptr_t)action_mask) & 15) == 0)
      hipLaunchKernelGGL(count_kernel<true>, grid, dim3(256), 0, s, T, n_traj, traj_id,
                         action_mask, seq_count, err);
    else
      hipLaunchKernelGGL(count_kernel<false>, grid, dim3(256), 0, s, T, n_traj, traj_id,
                         action_mask, seq_count, err);
    const int64_t blocks = cdiv<int64_t>(T, 256);
    hipLaunchKernelGGL(seq_weight_kernel, dim3((unsigned)(blocks < 1024 ? blocks : 1024)),
                       dim3(256), 0, s, T, n_traj, traj_id, action_mask,
                       (const int32_t*)seq_count, token_weight);
  }
  return hip_status(hipGetLastError());
}
