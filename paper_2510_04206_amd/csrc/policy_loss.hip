// Fused LM-head + token log-probability + clipped policy-gradient loss, forward
// and backward, over a packed micro-batch (AgentRL App. B.1 token-level
// factorisation; App. B.2 PPO/GRPO clipped surrogate; App. A DAPO decoupled
// clip bounds and token-level normalisation).
//
// Forward:  compact the action tokens -> logits H_act W^T by 256 x 256 tiles on
//           the matrix cores with a per-tile max / sum-exp epilogue (logits are
//           never written) -> merge the vocabulary tiles into lse -> logp,
//           ratio, clipped surrogate, fixed-order loss sum.
// Backward: recompute the logit tiles, form G = dL/dz in bf16 (one stage-tiled
//           layout, which dW reads transposed), then dW = G^T H and dH = G W on
//           the matrix cores; the vocabulary is processed in chunks that bound
//           the G buffer.
#include <math.h>

#include "../../include/agrl.h"
#include "common.hpp"
#include "gemm.hpp"

namespace agrl {
namespace {

constexpr int kScanTile = 4096;          // tokens per block of the compaction scan
constexpr int kScanThreads = 256;
constexpr int kScanPer = kScanTile / kScanThreads;   // 16 tokens per thread
constexpr int kRowPad = 256;             // compacted rows are padded to the GEMM tile
constexpr int kMergeRows = 64;         // action tokens per merge block

__host__ __device__ inline int64_t round_up(int64_t a, int64_t b) { return (a + b - 1) / b * b; }

// ------------------------------------------------------------------ compaction
__global__ __launch_bounds__(kScanThreads) void scan_count_kernel(int64_t T,
                                                                  const uint8_t* __restrict__ mask,
                                                                  int32_t* blk_cnt) {
  __shared__ int wsum[kScanThreads / 64];
  const int64_t base = (int64_t)blockIdx.x * kScanTile + threadIdx.x * kScanPer;
  int c = 0;
  for (int i = 0; i < kScanPer; ++i) {
    const int64_t t = base + i;
    if (t < T) c += mask[t] != 0;
  }
  for (int o = 32; o >= 1; o >>= 1) c += __shfl_xor(c, o);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    int s = 0;
    for (int w = 0; w < kScanThreads / 64; ++w) s += wsum[w];
    blk_cnt[blockIdx.x] = s;
  }
}

// Single block: exclusive offsets of the scan blocks, the action count, and
// the max_act check (an overflow zeroes the count and flags the call).
__global__ __launch_bounds__(1024) void scan_offsets_kernel(int32_t nblk,
                                                            const int32_t* __restrict__ blk_cnt,
                                                            int32_t* blk_off, int32_t* ctrl,
                                                            int64_t max_act, int* err) {
  __shared__ int wsum[16];
  __shared__ int carry;
  if (threadIdx.x == 0) carry = 0;
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int base = 0; base < nblk; base += 1024) {
    const int i = base + threadIdx.x;
    const int v = i < nblk ? blk_cnt[i] : 0;
    int incl = v;   // inclusive prefix within the wave
    for (int o = 1; o < 64; o <<= 1) {
      const int u = __shfl_up(incl, o);
      if (lane >= o) incl += u;
    }
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    int before = carry;
    for (int w = 0; w < wave; ++w) before += wsum[w];
    if (i < nblk) blk_off[i] = before + incl - v;
    __syncthreads();
    if (threadIdx.x == 1023) carry = before + incl;
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const int total = carry;
    if ((int64_t)total > max_act) {
      set_error(err, ERR_MAX_ACT);
      ctrl[0] = 0;
      ctrl[1] = 1;      // loss becomes NaN
    } else {
      ctrl[0] = total;
      ctrl[1] = 0;
    }
    ctrl[2] = total;
    ctrl[3] = 0;        // set by the scatter when an action token's id is out of range
  }
}

struct ScatterArgs {
  int64_t T;
  int32_t V;
  int32_t nblk;
  const uint8_t* mask;
  const int32_t* token_id;
  const float* adv_tok;
  const float* old_logp;
  const float* lse_in;      // backward only
  const float* logp_in;     // backward only
  const int32_t* blk_off;
  const int32_t* ctrl;
  int32_t* bad_id;          // ctrl[3]: 1 once an action token's id is out of range
  int64_t cap;              // rows allocated for compacted arrays
  int32_t* idx;
  int32_t* y_act;
  float* adv_act;
  float* old_act;
  float* lse_act;           // backward only
  float* gs_act;            // backward only: dL/dlogp / temperature
  float* logp_out;          // forward only: zeroed on masked tokens
  float* lse_out;
  const float* ref_logp;    // nullable: reference log-probs of the KL penalty
  const float* token_weight;  // nullable: per-token loss weights
  float* ref_act;           // forward only: compacted ref_logp / weights
  float* w_act;
  float kl_beta;
  int32_t kl_est;
  float eps_lo, eps_hi;
  float grad_loss;
  int64_t n_norm;
  float inv_temp;
  int* err;
};

__global__ __launch_bounds__(kScanThreads) void scan_scatter_kernel(ScatterArgs a) {
  __shared__ int wsum[kScanThreads / 64];
  const int64_t base = (int64_t)blockIdx.x * kScanTile + threadIdx.x * kScanPer;
  uint8_t m[kScanPer];
  int c = 0;
  for (int i = 0; i < kScanPer; ++i) {
    const int64_t t = base + i;
    m[i] = (t < a.T) ? (a.mask[t] != 0) : 0;
    c += m[i];
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int incl = c;
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(incl, o);
    if (lane >= o) incl += u;
  }
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  int pos = a.blk_off[blockIdx.x] + incl - c;
  for (int w = 0; w < wave; ++w) pos += wsum[w];
  const bool ok = a.ctrl[1] == 0;
  const int n_act = a.ctrl[2];
  const float N = a.n_norm > 0 ? (float)a.n_norm : (float)n_act;
  for (int i = 0; i < kScanPer; ++i) {
    const int64_t t = base + i;
    if (t >= a.T) break;
    if (!m[i]) {
      if (a.logp_out) {
        a.logp_out[t] = 0.0f;
        a.lse_out[t] = 0.0f;
      }
      continue;
    }
    const int y_in = a.token_id[t];
    // an id outside the vocabulary poisons the call: the token is kept with
    // id -1 (it matches no logit), its logp / lse become NaN in the merge, its
    // logit-gradient row NaN in the backward, and the loss NaN
    const bool bad = y_in < 0 || y_in >= a.V;
    const int y = bad ? -1 : y_in;
    if (bad) {
      set_error(a.err, ERR_TOKEN_ID);
      *a.bad_id = 1;
    }
    if (ok && pos < a.cap) {
      a.idx[pos] = (int32_t)t;
      a.y_act[pos] = y;
      // the forward-only log-prob pass has neither (its merge then forms a zero surrogate)
      const float adv = a.adv_tok ? a.adv_tok[t] : 0.0f;
      const float old = a.old_logp ? a.old_logp[t] : 0.0f;
      a.adv_act[pos] = adv;
      a.old_act[pos] = old;
      if (a.gs_act) {
        // dL/dlogp of -w (min(rho A, clip(rho) A) - beta KL), w = 1/N or the
        // token's weight: the unclipped branch's derivative, or 0 where the
        // clipped branch is the active minimum, plus w beta dKL/dlogp.
        const float lp = a.logp_in[t];
        const float rho = expf(lp - old);
        const bool cut = (adv > 0.0f && rho > 1.0f + a.eps_hi) || (adv < 0.0f && rho < 1.0f - a.eps_lo);
        const float scale = a.token_weight ? a.grad_loss * a.token_weight[t] : a.grad_loss / N;
        float g = cut ? 0.0f : -scale * adv * rho;
        if (a.kl_beta != 0.0f) {
          // k3: dKL/dl = 1 - exp(r - l) = -expm1(r - l); k1: 1
          const float dkl = a.kl_est == 1 ? 1.0f : -expm1f(a.ref_logp[t] - lp);
          g += scale * a.kl_beta * dkl;
        }
        a.lse_act[pos] = a.lse_in[t];
        a.gs_act[pos] = bad ? NAN : g * a.inv_temp;
      } else {
        a.ref_act[pos] = a.ref_logp ? a.ref_logp[t] : 0.0f;
        a.w_act[pos] = a.token_weight ? a.token_weight[t] : 0.0f;
      }
    }
    ++pos;
  }
}

// H_act[n] = H[idx[n]] for n < n_act, zero rows up to the next multiple of 256.
__global__ __launch_bounds__(256) void gather_rows_kernel(const uint8_t* __restrict__ H,
                                                          int64_t row_bytes,
                                                          const int32_t* __restrict__ idx,
                                                          const int32_t* ctrl, uint8_t* H_act) {
  const int n_act = ctrl[0];
  const int64_t rows = round_up(n_act, kRowPad);
  const int64_t chunks = row_bytes / 16;
  for (int64_t n = blockIdx.x; n < rows; n += gridDim.x) {
    u32x4* dst = (u32x4*)(H_act + n * row_bytes);
    if (n < n_act) {
      const u32x4* src = (const u32x4*)(H + (int64_t)idx[n] * row_bytes);
      for (int64_t c = threadIdx.x; c < chunks; c += blockDim.x) dst[c] = src[c];
    } else {
      for (int64_t c = threadIdx.x; c < chunks; c += blockDim.x) dst[c] = u32x4{0, 0, 0, 0};
    }
  }
}

// dst[c][r] = src[r][c]; rows in [n_rows, n_rows_pad) are written as 0.
// n_rows comes from ctrl[0] (rounded up to 256 for the padded extent) when
// ctrl is given.  64 x 64 element tiles through LDS.  With `tiled`, dst is
// stage-tiled (tiled_index, K = r padded to ld_dst) instead of row-major.
template <typename T>
__global__ __launch_bounds__(256) void transpose_kernel(const T* __restrict__ src, int64_t ld_src,
                                                        T* dst, int64_t ld_dst, int64_t n_rows,
                                                        int64_t n_rows_pad, int64_t n_cols,
                                                        const int32_t* ctrl, int32_t tiled) {
  __shared__ T tile[64][65];
  if (ctrl) {
    n_rows = ctrl[0];
    n_rows_pad = round_up(n_rows, kRowPad);
  }
  const int64_t r0 = (int64_t)blockIdx.x * 64, c0 = (int64_t)blockIdx.y * 64;
  if (r0 >= n_rows_pad) return;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int k = 0; k < 16; ++k) {
    const int rr = ty + 4 * k;
    const int64_t r = r0 + rr, c = c0 + tx;
    T v = T(0);
    if (r < n_rows && c < n_cols) v = src[r * ld_src + c];
    tile[rr][tx] = v;
  }
  __syncthreads();
  for (int k = 0; k < 16; ++k) {
    const int cc = ty + 4 * k;
    const int64_t c = c0 + cc, r = r0 + tx;
    if (c < n_cols && r < n_rows_pad)
      dst[tiled ? tiled_index(c, r, ld_dst) : c * ld_dst + r] = tile[tx][cc];
  }
}

// bf16 (2-byte) variant of transpose_kernel with 16-byte global accesses: each
// 64 x 64 tile is read as 8-element row chunks, written to LDS transposed
// (66-element rows: the 16-bit stores of a wave hit distinct banks), and read
// back as 8-element chunks of the output rows.  Same arguments and padding
// rules; d (the source row length) is a multiple of 64.
__global__ __launch_bounds__(256) void transpose16_kernel(const uint16_t* __restrict__ src,
                                                          int64_t ld_src, uint16_t* dst,
                                                          int64_t ld_dst, int64_t n_rows,
                                                          int64_t n_rows_pad, int64_t n_cols,
                                                          const int32_t* ctrl, int32_t tiled) {
  constexpr int P = 66;
  __shared__ uint16_t tile_t[64 * P];
  if (ctrl) {
    n_rows = ctrl[0];
    n_rows_pad = round_up(n_rows, kRowPad);
  }
  const int64_t r0 = (int64_t)blockIdx.x * 64, c0 = (int64_t)blockIdx.y * 64;
  if (r0 >= n_rows_pad) return;
  for (int k = 0; k < 2; ++k) {
    const int id = threadIdx.x + 256 * k;
    const int rr = id >> 3, c8 = id & 7;
    const int64_t r = r0 + rr;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (r < n_rows) v = *(const u32x4*)(src + r * ld_src + c0 + 8 * c8);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      tile_t[(8 * c8 + 2 * e) * P + rr] = (uint16_t)v[e];
      tile_t[(8 * c8 + 2 * e + 1) * P + rr] = (uint16_t)(v[e] >> 16);
    }
  }
  __syncthreads();
  for (int k = 0; k < 2; ++k) {
    const int id = threadIdx.x + 256 * k;
    const int c = id >> 3, r8 = id & 7;
    const uint32_t* t32 = (const uint32_t*)(tile_t + c * P + 8 * r8);   // 4-byte aligned
    const u32x4 v = {t32[0], t32[1], t32[2], t32[3]};
    const int64_t oc = c0 + c, orr = r0 + 8 * r8;
    if (oc < n_cols && orr < n_rows_pad)
      *(u32x4*)(dst + (tiled ? tiled_index(oc, orr, ld_dst) : oc * ld_dst + orr)) = v;
  }
}

// ------------------------------------------------------------------ forward epilogue
struct MergeArgs {
  const int32_t* ctrl;
  int32_t tiles_v;
  const f32x2* part;
  int64_t ld_part;
  const float* zy;
  const int32_t* y_act;    // -1 marks an action token whose id was out of range
  const float* old_act;
  const float* adv_act;
  const float* ref_act;
  const float* w_act;
  const int32_t* idx;
  float eps_lo, eps_hi;
  float kl_beta;
  int32_t kl_est;
  int32_t weighted;        // loss partials are w_n f_n (else f_n, divided by N at the end)
  float* logp_out;
  float* lse_out;
  double* blk_sum;
  long long* blk_clip;     // [2 * blocks]
};

// 64 action tokens per block.  Each of the 4 waves folds a quarter of the
// vocabulary-tile partials of its lane's token with the online log-sum-exp
// update; wave 0 combines the four, then forms logp, rho and the clipped
// surrogate and writes the block's fixed-order partial sums.
__global__ __launch_bounds__(256) void merge_loss_kernel(MergeArgs a) {
  __shared__ f32x2 wpart[4][kMergeRows];
  const int n_act = a.ctrl[0];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = blockIdx.x * kMergeRows + lane;
  float m = -INFINITY, s = 0.0f;
  if (n < n_act) {
    for (int t = wave; t < a.tiles_v; t += 4) {
      const f32x2 p = a.part[(int64_t)t * a.ld_part + n];
      const float mn = fmaxf(m, p.x);
      s = s * expf(m - mn) + p.y * expf(p.x - mn);
      m = mn;
    }
  }
  wpart[wave][lane] = f32x2{m, s};
  __syncthreads();
  if (wave != 0) return;
  double sv = 0.0;
  long long hi = 0, lo = 0;
  if (n < n_act) {
    float mm = -INFINITY;
    for (int w = 0; w < 4; ++w) mm = fmaxf(mm, wpart[w][lane].x);
    float sum = 0.0f;
    for (int w = 0; w < 4; ++w)
      if (wpart[w][lane].y > 0.0f) sum += wpart[w][lane].y * expf(wpart[w][lane].x - mm);
    const bool bad = a.y_act[n] < 0;
    const float lse = bad ? NAN : mm + logf(sum);
    const float logp = bad ? NAN : a.zy[n] - lse;
    const float A = a.adv_act[n];
    const float rho = expf(logp - a.old_act[n]);
    const float rc = fminf(fmaxf(rho, 1.0f - a.eps_lo), 1.0f + a.eps_hi);
    float f = fminf(rho * A, rc * A);
    if (a.kl_beta != 0.0f) {
      // k3: exp(u) - u - 1 = expm1(u) - u with u = r - l (no cancellation near u = 0)
      const float u = a.ref_act[n] - logp;
      f -= a.kl_beta * (a.kl_est == 1 ? -u : expm1f(u) - u);
    }
    sv = a.weighted ? (double)a.w_act[n] * (double)f : (double)f;
    hi = (A > 0.0f && rho > 1.0f + a.eps_hi);
    lo = (A < 0.0f && rho < 1.0f - a.eps_lo);
    const int t = a.idx[n];
    a.logp_out[t] = logp;
    a.lse_out[t] = lse;
  }
  for (int o = 32; o >= 1; o >>= 1) {
    sv += __shfl_xor(sv, o);
    hi += __shfl_xor(hi, o);
    lo += __shfl_xor(lo, o);
  }
  if (lane == 0) {
    a.blk_sum[blockIdx.x] = sv;
    a.blk_clip[2 * blockIdx.x] = hi;
    a.blk_clip[2 * blockIdx.x + 1] = lo;
  }
}

__global__ __launch_bounds__(256) void finalize_loss_kernel(int32_t nblk, const double* blk_sum,
                                                            const long long* blk_clip,
                                                            const int32_t* ctrl, int64_t n_norm,
                                                            int32_t weighted, float* loss,
                                                            int64_t* n_clip) {
  __shared__ double ssum[256];
  __shared__ long long shi[256], slo[256];
  double s = 0.0;
  long long hi = 0, lo = 0;
  for (int b = threadIdx.x; b < nblk; b += 256) {
    s += blk_sum[b];
    hi += blk_clip[2 * b];
    lo += blk_clip[2 * b + 1];
  }
  ssum[threadIdx.x] = s;
  shi[threadIdx.x] = hi;
  slo[threadIdx.x] = lo;
  __syncthreads();
  for (int w = 128; w >= 1; w >>= 1) {
    if (threadIdx.x < w) {
      ssum[threadIdx.x] += ssum[threadIdx.x + w];
      shi[threadIdx.x] += shi[threadIdx.x + w];
      slo[threadIdx.x] += slo[threadIdx.x + w];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const int n_act = ctrl[0];
    const double N = n_norm > 0 ? (double)n_norm : (double)n_act;
    float L = weighted ? (float)(-ssum[0]) : (N > 0 ? (float)(-ssum[0] / N) : 0.0f);
    if (ctrl[1] || ctrl[3]) L = NAN;
    *loss = L;
    if (n_clip) {
      n_clip[0] = shi[0];
      n_clip[1] = slo[0];
    }
  }
}

__global__ void zero_loss_kernel(float* loss, int64_t* n_clip) {
  *loss = 0.0f;
  if (n_clip) {
    n_clip[0] = 0;
    n_clip[1] = 0;
  }
}

__global__ __launch_bounds__(256) void zero_masked_rows_kernel(int64_t T, int32_t d,
                                                               const uint8_t* __restrict__ mask,
                                                               float* dH) {
  for (int64_t t = blockIdx.x; t < T; t += gridDim.x) {
    if (mask[t]) continue;
    f32x4* row = (f32x4*)(dH + t * d);
    for (int c = threadIdx.x; c < d / 4; c += blockDim.x) row[c] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
}

__global__ __launch_bounds__(256) void zero_f32_kernel(float* p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0.0f;
}

// ------------------------------------------------------------------ host side
int fail(int code, const char* msg) {
  set_last_error(msg);
  return code;
}

struct Layout {
  int64_t T, A_pad, V_pad, Vc;
  int32_t d, V, esize, nblk, tiles_v, merge_blocks;
  size_t ctrl, blk_cnt, blk_off, idx, y_act, adv_act, old_act, ref_act, w_act, lse_act, gs_act,
      zy, blk_sum,
      blk_clip, H_act, part, Ht, Wt, G, Gt, fwd_total, total;
};

constexpr int64_t kDefaultChunkBytes = (int64_t)4 << 30;

bool make_layout(int64_t T, int64_t max_act, int32_t d, int32_t V, int32_t dtype,
                 const agrl_options& o, Layout* L) {
  if (T < 0 || d <= 0 || V <= 0 || (dtype != AGRL_BF16 && dtype != AGRL_F32)) return false;
  if (max_act <= 0 || max_act > T) max_act = T;
  L->T = T;
  L->d = d;
  L->V = V;
  L->esize = dtype == AGRL_BF16 ? 2 : 4;
  L->A_pad = round_up(max_act > 0 ? max_act : 1, kRowPad);
  L->V_pad = round_up(V, kRowPad);
  L->nblk = (int32_t)((T + kScanTile - 1) / kScanTile);
  if (L->nblk < 1) L->nblk = 1;
  L->tiles_v = (int32_t)(L->V_pad / GBN);
  L->merge_blocks = (int32_t)(L->A_pad / kMergeRows);
  // vocabulary chunk of the backward: the widest multiple of 256 whose logit
  // gradient buffers (bf16: G, read transposed by dW; fp32: G and G^T) fit the
  // budget, then evened out over the chunks this needs
  const int64_t budget = o.g_chunk_bytes > 0 ? o.g_chunk_bytes : kDefaultChunkBytes;
  const int64_t g_copies = dtype == AGRL_BF16 ? 1 : 2;
  int64_t vc_max = budget / (g_copies * L->A_pad * L->esize) / kRowPad * kRowPad;
  if (vc_max < kRowPad) vc_max = kRowPad;
  const int64_t n_chunks = (L->V_pad + vc_max - 1) / vc_max;
  L->Vc = round_up((V + n_chunks - 1) / n_chunks, kRowPad);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off += (bytes + 255) / 256 * 256;
    return at;
  };
  const size_t A = (size_t)L->A_pad;
  L->ctrl = take(256);
  L->blk_cnt = take(sizeof(int32_t) * L->nblk);
  L->blk_off = take(sizeof(int32_t) * L->nblk);
  L->idx = take(4 * A);
  L->y_act = take(4 * A);
  L->adv_act = take(4 * A);
  L->old_act = take(4 * A);
  L->ref_act = take(4 * A);
  L->w_act = take(4 * A);
  L->lse_act = take(4 * A);
  L->gs_act = take(4 * A);
  L->zy = take(4 * A);
  L->blk_sum = take(sizeof(double) * L->merge_blocks);
  L->blk_clip = take(2 * sizeof(long long) * L->merge_blocks);
  L->H_act = take(A * d * L->esize);
  // the forward's partials and the backward's buffers share one region
  const size_t shared_at = off;
  L->part = take((size_t)L->tiles_v * A * 8);
  const size_t fwd_end = off;
  L->fwd_total = fwd_end;
  off = shared_at;
  // H^T and W^T: d rows padded to a whole 256-row tile (bf16 stage-tiled layout)
  const size_t d_pad = (size_t)round_up(d, kRowPad);
  L->Ht = take(d_pad * A * L->esize);
  L->Wt = take(d_pad * L->V_pad * L->esize);
  L->G = take(A * (size_t)L->Vc * L->esize);
  L->Gt = dtype == AGRL_BF16 ? L->G : take((size_t)L->Vc * A * L->esize);
  if (fwd_end > off) off = fwd_end;
  L->total = off;
  return true;
}

struct Common {
  int64_t T, max_act;
  int32_t d, V, dtype;
  float eps_lo, eps_hi, inv_temp;
  agrl_options o;
};

int validate(const char* fn, int64_t T, int64_t max_act, int32_t d, int32_t V, int32_t dtype,
             const void* H, const void* W, const int32_t* token_id, const uint8_t* mask,
             const float* adv, const float* old, float eps_lo, float eps_hi, int64_t n_norm,
             const agrl_options* opt, void* ws, size_t ws_bytes, Common* c,
             bool loss_inputs = true) {
  char buf[200];
  auto bad = [&](int code, const char* what) {
    snprintf(buf, sizeof buf, "%s: %s", fn, what);
    return fail(code, buf);
  };
  if (dtype != AGRL_BF16 && dtype != AGRL_F32) return bad(AGRL_E_DTYPE, "dtype must be AGRL_BF16 or AGRL_F32");
  if (T < 0) return bad(AGRL_E_SHAPE, "T < 0");
  if (T > ((int64_t)1 << 31) - kScanTile) return bad(AGRL_E_SHAPE, "T too large");
  if (d <= 0 || V <= 0) return bad(AGRL_E_SHAPE, "d and V must be positive");
  if (d % 64 != 0) return bad(AGRL_E_UNSUPPORTED, "d must be a multiple of 64");
  if (n_norm < 0) return bad(AGRL_E_SHAPE, "n_norm < 0");
  if (!(eps_lo >= 0.0f && eps_lo < 1.0f) || !(eps_hi >= 0.0f) || !isfinite(eps_hi))
    return bad(AGRL_E_FLAGS, "clip bounds must satisfy 0 <= low < 1 and 0 <= high < inf");
  agrl_options o = {};
  if (opt) o = *opt;
  if (!(o.temperature >= 0.0f) || !isfinite(o.temperature))
    return bad(AGRL_E_FLAGS, "temperature must be finite and >= 0");
  if (o.dw_accumulate != 0 && o.dw_accumulate != 1) return bad(AGRL_E_FLAGS, "dw_accumulate must be 0 or 1");
  if (o.g_chunk_bytes < 0) return bad(AGRL_E_FLAGS, "g_chunk_bytes < 0");
  if (!isfinite(o.kl_beta)) return bad(AGRL_E_FLAGS, "kl_beta must be finite");
  if (o.kl_estimator != 0 && o.kl_estimator != 1) return bad(AGRL_E_FLAGS, "kl_estimator must be 0 or 1");
  if (loss_inputs && o.kl_beta != 0.0f && T > 0 && !o.ref_logp)
    return bad(AGRL_E_NULL, "kl_beta != 0 needs ref_logp");
  if (T > 0 && (!H || !token_id || !mask || (loss_inputs && (!adv || !old))))
    return bad(AGRL_E_NULL, "input pointer is NULL");
  if (!W) return bad(AGRL_E_NULL, "W is NULL");
  if (max_act <= 0 || max_act > T) max_act = T;
  // every tile row offset and the G buffers use 32-bit row indices
  // operand rows are addressed as 32-bit offsets within a 256-row tile, so a row
  // of any operand (d, V or the padded action count, in elements) stays below 8M
  // (this also bounds dW's transposed read of G: three block columns of at most
  // 2^15 blocks of 32 KiB)
  if (round_up(max_act > 0 ? max_act : 1, kRowPad) > ((int64_t)1 << 23)) return bad(AGRL_E_SHAPE, "max_act too large");
  if (round_up(V, kRowPad) > ((int64_t)1 << 23) || d > (1 << 23)) return bad(AGRL_E_SHAPE, "V or d too large");
  Layout L;
  make_layout(T, max_act, d, V, dtype, o, &L);
  const size_t need = loss_inputs ? L.total : L.fwd_total;
  if (T > 0 && (!ws || ws_bytes < need)) return bad(AGRL_E_WORKSPACE, "workspace missing or too small");
  if ((((uintptr_t)H | (uintptr_t)W | (uintptr_t)ws) & 15) != 0)
    return bad(AGRL_E_SHAPE, "H, W and workspace must be 16-byte aligned");
  c->T = T;
  c->max_act = max_act;
  c->d = d;
  c->V = V;
  c->dtype = dtype;
  c->eps_lo = eps_lo;
  c->eps_hi = eps_hi;
  c->inv_temp = o.temperature == 0.0f ? 1.0f : 1.0f / o.temperature;
  c->o = o;
  return AGRL_OK;
}

enum Phase { PH_FWD = 0, PH_RECOMPUTE = 1, PH_DW = 2, PH_DH = 3 };

__global__ void zero_queue_kernel(int32_t* q) {
  if (threadIdx.x < 16) q[threadIdx.x] = 0;
}

// Launch n (1 or 2) independent products.  bf16: one persistent launch of the
// pipelined kernel with its tile queues reset first; fp32: one simple launch
// per product.  The phase's events bracket the whole launch (a second phase
// slot, when given, is recorded empty).
template <typename T, class Epi>
void launch_gemm(const GemmShape* g, const Epi* e, int n, int max_tiles, int32_t* queue,
                 const agrl_options& o, Phase ph, int ph2, hipStream_t s) {
  int grid = device_cu_count();
  if (max_tiles < grid) grid = max_tiles < 1 ? 1 : max_tiles;
  hipEvent_t* ev = (hipEvent_t*)o.phase_events;
  if constexpr (std::is_same<T, __bf16>::value) {
    GemmBatch<Epi> b;
    for (int i = 0; i < 2; ++i) {
      b.g[i] = g[i < n ? i : 0];
      b.e[i] = e[i < n ? i : 0];
    }
    b.n = n;
    b.queue = queue;
    // every K a whole number of stage pairs (device-read ones are rounded up
    // in the kernel, their operands being zero-padded to 256)
    bool even = true, atr = false;
    for (int i = 0; i < n; ++i) {
      even = even && (g[i].k_dev != nullptr || g[i].K % (2 * KStage<T>::BK) == 0);
      atr = atr || g[i].a_trans;
    }
    hipLaunchKernelGGL(zero_queue_kernel, dim3(1), dim3(64), 0, s, queue);
    if (ev) hipEventRecord(ev[2 * ph], s);
    // The bf16 store launch is the backward's dH + dW: its operands are
    // stage-tiled, dW reads G transposed, and both K extents are whole stage
    // pairs (the vocabulary chunk rounded up to 128, the device-read token count
    // rounded up in the kernel), so it always runs the 16 x 16 loop.
    if constexpr (std::is_same<Epi, EpiStore>::value) {
      (void)atr;
      (void)even;
      hipLaunchKernelGGL((gemm_bf16_kernel<Epi, true, true, true>), dim3(grid), dim3(GEMM_THREADS),
                         0, s, b);
    } else {
      if (even)
        hipLaunchKernelGGL((gemm_bf16_kernel<Epi, true, false, true>), dim3(grid),
                           dim3(GEMM_THREADS), 0, s, b);
      else
        hipLaunchKernelGGL((gemm_bf16_kernel<Epi, false, false>), dim3(grid), dim3(GEMM_THREADS),
                           0, s, b);
    }
    if (ev) hipEventRecord(ev[2 * ph + 1], s);
    if (ev && ph2 >= 0) {
      hipEventRecord(ev[2 * ph2], s);
      hipEventRecord(ev[2 * ph2 + 1], s);
    }
  } else {
    for (int i = 0; i < n; ++i) {
      // with two problems the first is dH (slot ph2) and the second dW (slot ph)
      const int p = (n == 2 && ph2 >= 0) ? (i == 0 ? ph2 : ph) : ph;
      if (ev) hipEventRecord(ev[2 * p], s);
      hipLaunchKernelGGL((gemm_nt_kernel<T, Epi>), dim3(grid), dim3(GEMM_THREADS), 0, s, g[i],
                         e[i]);
      if (ev) hipEventRecord(ev[2 * p + 1], s);
    }
  }
}

int compact(const Common& c, const Layout& L, uint8_t* ws, const uint8_t* mask,
            const int32_t* token_id, const float* adv, const float* old, const float* lse_in,
            const float* logp_in, float grad_loss, int64_t n_norm, float* logp_out,
            float* lse_out, const void* H, int* err, hipStream_t s) {
  int32_t* ctrl = (int32_t*)(ws + L.ctrl);
  hipLaunchKernelGGL(scan_count_kernel, dim3(L.nblk), dim3(kScanThreads), 0, s, c.T, mask,
                     (int32_t*)(ws + L.blk_cnt));
  hipLaunchKernelGGL(scan_offsets_kernel, dim3(1), dim3(1024), 0, s, L.nblk,
                     (const int32_t*)(ws + L.blk_cnt), (int32_t*)(ws + L.blk_off), ctrl,
                     c.max_act, err);
  ScatterArgs a;
  a.T = c.T;
  a.V = c.V;
  a.nblk = L.nblk;
  a.mask = mask;
  a.token_id = token_id;
  a.adv_tok = adv;
  a.old_logp = old;
  a.lse_in = lse_in;
  a.logp_in = logp_in;
  a.blk_off = (const int32_t*)(ws + L.blk_off);
  a.ctrl = ctrl;
  a.bad_id = ctrl + 3;
  a.cap = L.A_pad;
  a.idx = (int32_t*)(ws + L.idx);
  a.y_act = (int32_t*)(ws + L.y_act);
  a.adv_act = (float*)(ws + L.adv_act);
  a.old_act = (float*)(ws + L.old_act);
  a.lse_act = lse_in ? (float*)(ws + L.lse_act) : nullptr;
  a.gs_act = lse_in ? (float*)(ws + L.gs_act) : nullptr;
  a.logp_out = logp_out;
  a.lse_out = lse_out;
  a.ref_logp = c.o.kl_beta != 0.0f ? c.o.ref_logp : nullptr;
  a.token_weight = c.o.token_weight;
  a.ref_act = (float*)(ws + L.ref_act);
  a.w_act = (float*)(ws + L.w_act);
  a.kl_beta = c.o.kl_beta;
  a.kl_est = c.o.kl_estimator;
  a.eps_lo = c.eps_lo;
  a.eps_hi = c.eps_hi;
  a.grad_loss = grad_loss;
  a.n_norm = n_norm;
  a.inv_temp = c.inv_temp;
  a.err = err;
  hipLaunchKernelGGL(scan_scatter_kernel, dim3(L.nblk), dim3(kScanThreads), 0, s, a);
  const int64_t rows = L.A_pad;
  const int grid = (int)(rows < 4096 ? rows : 4096);
  hipLaunchKernelGGL(gather_rows_kernel, dim3(grid), dim3(256), 0, s, (const uint8_t*)H,
                     (int64_t)c.d * L.esize, (const int32_t*)(ws + L.idx), (const int32_t*)ctrl,
                     ws + L.H_act);
  return AGRL_OK;
}

template <typename T>
void fwd_gemm(const Common& c, const Layout& L, uint8_t* ws, const void* W, hipStream_t s) {
  const int32_t* n_act = (const int32_t*)(ws + L.ctrl);
  const int max_tiles = (int)(L.A_pad / GBM) * L.tiles_v;
  GemmShape g = {};
  g.K = c.d;
  g.group_m = 8;
  if constexpr (std::is_same<T, __bf16>::value) {
    // transposed tile (rows: vocabulary, columns: action tokens), so that the
    // log-sum-exp over the vocabulary reduces mostly inside each lane
    g.A = W;
    g.lda = c.d;
    g.M = c.V;
    g.B = ws + L.H_act;
    g.ldb = c.d;
    g.N = (int32_t)L.A_pad;
    g.n_dev = n_act;
    EpiLseCols e;
    e.y = (const int32_t*)(ws + L.y_act);
    e.part = (f32x2*)(ws + L.part);
    e.ld_part = L.A_pad;
    e.zy = (float*)(ws + L.zy);
    e.scale = c.inv_temp;
    launch_gemm<T>(&g, &e, 1, max_tiles, (int32_t*)(ws + L.ctrl + 64), c.o, PH_FWD, -1, s);
  } else {
    g.A = ws + L.H_act;
    g.lda = c.d;
    g.B = W;
    g.ldb = c.d;
    g.m_dev = n_act;
    g.N = c.V;
    EpiLsePartial e;
    e.y = (const int32_t*)(ws + L.y_act);
    e.part = (f32x2*)(ws + L.part);
    e.ld_part = L.A_pad;
    e.zy = (float*)(ws + L.zy);
    e.scale = c.inv_temp;
    launch_gemm<T>(&g, &e, 1, max_tiles, (int32_t*)(ws + L.ctrl + 64), c.o, PH_FWD, -1, s);
  }
}

template <typename T>
struct Storage {
  typedef uint16_t type;   // bf16 moved as raw bits
};
template <>
struct Storage<float> {
  typedef float type;
};

template <typename T>
void bwd_gemms(const Common& c, const Layout& L, uint8_t* ws, const void* W, float* dH, float* dW,
               hipStream_t s) {
  typedef typename Storage<T>::type S;
  const int32_t* ctrl = (const int32_t*)(ws + L.ctrl);
  T* Ht = (T*)(ws + L.Ht);
  T* Wt = (T*)(ws + L.Wt);
  T* G = (T*)(ws + L.G);
  T* Gt = (T*)(ws + L.Gt);   // fp32 only
  // H_act^T [d][A_pad] (zero beyond the action rows) and W^T [d][V_pad] (zero
  // beyond V); for bf16 both, and G, are stage-tiled: every stage of the two
  // products below is a contiguous 32 KiB block per operand tile (8 KiB in each
  // of four blocks for dW's transposed read of G)
  constexpr int32_t tiled = std::is_same<T, __bf16>::value ? 1 : 0;
  const dim3 gh((unsigned)(L.A_pad / 64), (unsigned)cdiv(c.d, 64));
  const dim3 gw((unsigned)(L.V_pad / 64), (unsigned)cdiv(c.d, 64));
  if constexpr (sizeof(S) == 2) {
    hipLaunchKernelGGL(transpose16_kernel, gh, dim3(256), 0, s, (const uint16_t*)(ws + L.H_act),
                       (int64_t)c.d, (uint16_t*)Ht, L.A_pad, (int64_t)0, (int64_t)0,
                       (int64_t)c.d, ctrl, tiled);
    hipLaunchKernelGGL(transpose16_kernel, gw, dim3(256), 0, s, (const uint16_t*)W, (int64_t)c.d,
                       (uint16_t*)Wt, L.V_pad, (int64_t)c.V, L.V_pad, (int64_t)c.d,
                       (const int32_t*)nullptr, tiled);
  } else {
    hipLaunchKernelGGL((transpose_kernel<S>), gh, dim3(256), 0, s, (const S*)(ws + L.H_act),
                       (int64_t)c.d, (S*)Ht, L.A_pad, (int64_t)0, (int64_t)0, (int64_t)c.d, ctrl,
                       tiled);
    hipLaunchKernelGGL((transpose_kernel<S>), gw, dim3(256), 0, s, (const S*)W, (int64_t)c.d,
                       (S*)Wt, L.V_pad, (int64_t)c.V, L.V_pad, (int64_t)c.d,
                       (const int32_t*)nullptr, tiled);
  }
  const int row_tiles = (int)(L.A_pad / GBM);
  const int d_tiles = cdiv(c.d, GBN);
  for (int64_t v0 = 0; v0 < c.V; v0 += L.Vc) {
    const int32_t nv = (int32_t)((c.V - v0) < L.Vc ? (c.V - v0) : L.Vc);
    const int nv_tiles = cdiv(nv, GBN);
    {  // logits of the chunk -> G (and G^T for fp32)
      GemmShape g = {};
      g.A = ws + L.H_act;
      g.lda = c.d;
      g.B = (const uint8_t*)W + v0 * c.d * (int64_t)sizeof(T);
      g.ldb = c.d;
      g.m_dev = ctrl;
      g.N = nv;
      g.K = c.d;
      // groups of 8 vocabulary tiles sweep every token tile: each W panel of the
      // chunk is read from memory once (the compacted H is small enough to stay
      // in the Infinity Cache), not once per group of 8 token tiles
      g.group_m = 8;
      g.group_cols = 1;
      EpiLogitGrad<T> e;
      e.y = (const int32_t*)(ws + L.y_act);
      e.lse = (const float*)(ws + L.lse_act);
      e.gs = (const float*)(ws + L.gs_act);
      e.G = G;
      e.ldg = tiled ? L.A_pad : L.Vc;
      e.Gt = tiled ? nullptr : Gt;
      e.ldgt = L.A_pad;
      e.scale = c.inv_temp;
      e.col0 = (int32_t)v0;
      launch_gemm<T>(&g, &e, 1, row_tiles * nv_tiles, (int32_t*)(ws + L.ctrl + 64), c.o,
                     PH_RECOMPUTE, -1, s);
    }
    {  // dH[idx] (+)= G W[v0 : v0 + nv] (K = the chunk's vocabulary columns) and
       // dW[v0 : v0 + nv] = G^T H_act (K = action tokens), one launch, dH first:
       // its tiles are the long ones.  bf16 G is column-block stage-tiled; dW
       // reads it transposed (fp32 reads the separate G^T)
      GemmShape g[2] = {};
      g[0].A = G;
      g[0].lda = tiled ? L.A_pad : L.Vc;
      // the chunk's first vocabulary column: a row offset, or whole 64-column blocks
      g[0].B = tiled ? (const void*)(Wt + v0 * 256) : (const void*)(Wt + v0);
      g[0].ldb = L.V_pad;
      g[0].a_tiled = tiled ? 2 : 0;
      g[0].b_tiled = tiled;
      g[0].m_dev = ctrl;
      g[0].N = c.d;
      // (bf16: a whole number of stage pairs; G and W^T are zero up to Vc and V_pad)
      g[0].K = (int32_t)round_up(nv, (tiled ? 2 : 1) * KStage<T>::BK);
      g[0].group_m = 8;
      g[1].A = tiled ? G : Gt;
      g[1].lda = L.A_pad;
      g[1].B = Ht;
      g[1].ldb = L.A_pad;
      g[1].a_tiled = tiled ? 2 : 0;
      g[1].a_trans = tiled;
      g[1].b_tiled = tiled;
      g[1].M = nv;
      g[1].N = c.d;
      g[1].k_dev = ctrl;
      g[1].group_m = 8;
      EpiStore e[2];
      e[0].out = dH;
      e[0].ldo = c.d;
      e[0].row_map = (const int32_t*)(ws + L.idx);
      e[0].accumulate = v0 > 0;
      e[1].out = dW + v0 * c.d;
      e[1].ldo = c.d;
      e[1].row_map = nullptr;
      e[1].accumulate = c.o.dw_accumulate;
      launch_gemm<T>(g, e, 2, row_tiles * d_tiles + nv_tiles * d_tiles,
                     (int32_t*)(ws + L.ctrl + 64), c.o, PH_DW, PH_DH, s);
    }
  }
}

}  // namespace
}  // namespace agrl

extern "C" int64_t agrl_policy_loss_vocab_chunk(int64_t T, int64_t max_act, int32_t d,
                                                int32_t V, int32_t dtype,
                                                const agrl_options* opt) {
  agrl_options o = {};
  if (opt) o = *opt;
  agrl::Layout L;
  if (T <= 0 || o.g_chunk_bytes < 0 || !agrl::make_layout(T, max_act, d, V, dtype, o, &L)) return 0;
  return L.Vc;
}

extern "C" size_t agrl_policy_loss_workspace_size(int64_t T, int64_t max_act, int32_t d,
                                                  int32_t V, int32_t dtype,
                                                  const agrl_options* opt) {
  agrl_options o = {};
  if (opt) o = *opt;
  agrl::Layout L;
  if (T <= 0 || o.g_chunk_bytes < 0 || !agrl::make_layout(T, max_act, d, V, dtype, o, &L)) return 0;
  return L.total;
}

extern "C" int agrl_policy_loss_fwd(int64_t T, int64_t max_act, int32_t d, int32_t V,
                                    int32_t dtype, const void* H, const void* W,
                                    const int32_t* token_id, const uint8_t* action_mask,
                                    const float* adv_tok, const float* old_logp,
                                    float clip_eps_low, float clip_eps_high, int64_t n_norm,
                                    const agrl_options* opt, void* workspace, size_t ws_bytes,
                                    float* loss, float* logp, float* lse, int64_t* n_clip,
                                    void* stream) {
  using namespace agrl;
  Common c;
  int rc = validate("agrl_policy_loss_fwd", T, max_act, d, V, dtype, H, W, token_id, action_mask,
                    adv_tok, old_logp, clip_eps_low, clip_eps_high, n_norm, opt, workspace,
                    ws_bytes, &c);
  if (rc) return rc;
  if (!loss || (T > 0 && (!logp || !lse))) return fail(AGRL_E_NULL, "agrl_policy_loss_fwd: output pointer is NULL");
  hipStream_t s = (hipStream_t)stream;
  int* err = device_error_ptr();
  if (!err) return hip_status(hipErrorInvalidSymbol);
  if (T == 0) {
    hipLaunchKernelGGL(zero_loss_kernel, dim3(1), dim3(1), 0, s, loss, n_clip);
    return hip_status(hipGetLastError());
  }
  Layout L;
  make_layout(T, c.max_act, d, V, dtype, c.o, &L);
  uint8_t* ws = (uint8_t*)workspace;
  compact(c, L, ws, action_mask, token_id, adv_tok, old_logp, nullptr, nullptr, 0.0f, n_norm,
          logp, lse, H, err, s);
  if (dtype == AGRL_BF16)
    fwd_gemm<__bf16>(c, L, ws, W, s);
  else
    fwd_gemm<float>(c, L, ws, W, s);
  MergeArgs m;
  m.ctrl = (const int32_t*)(ws + L.ctrl);
  m.tiles_v = L.tiles_v;
  m.part = (const f32x2*)(ws + L.part);
  m.ld_part = L.A_pad;
  m.zy = (const float*)(ws + L.zy);
  m.y_act = (const int32_t*)(ws + L.y_act);
  m.old_act = (const float*)(ws + L.old_act);
  m.adv_act = (const float*)(ws + L.adv_act);
  m.idx = (const int32_t*)(ws + L.idx);
  m.eps_lo = c.eps_lo;
  m.eps_hi = c.eps_hi;
  m.ref_act = (const float*)(ws + L.ref_act);
  m.w_act = (const float*)(ws + L.w_act);
  m.kl_beta = c.o.kl_beta;
  m.kl_est = c.o.kl_estimator;
  m.weighted = c.o.token_weight != nullptr;
  m.logp_out = logp;
  m.lse_out = lse;
  m.blk_sum = (double*)(ws + L.blk_sum);
  m.blk_clip = (long long*)(ws + L.blk_clip);
  hipLaunchKernelGGL(merge_loss_kernel, dim3(L.merge_blocks), dim3(256), 0, s, m);
  hipLaunchKernelGGL(finalize_loss_kernel, dim3(1), dim3(256), 0, s, L.merge_blocks,
                     (const double*)(ws + L.blk_sum), (const long long*)(ws + L.blk_clip),
                     (const int32_t*)(ws + L.ctrl), n_norm, (int32_t)(c.o.token_weight != nullptr),
                     loss, n_clip);
  return hip_status(hipGetLastError());
}

extern "C" size_t agrl_token_logprob_workspace_size(int64_t T, int64_t max_act, int32_t d,
                                                    int32_t V, int32_t dtype,
                                                    const agrl_options* opt) {
  agrl_options o = {};
  if (opt) o = *opt;
  agrl::Layout L;
  if (T <= 0 || o.g_chunk_bytes < 0 || !agrl::make_layout(T, max_act, d, V, dtype, o, &L)) return 0;
  return L.fwd_total;
}

extern "C" int agrl_token_logprob(int64_t T, int64_t max_act, int32_t d, int32_t V, int32_t dtype,
                                  const void* H, const void* W, const int32_t* token_id,
                                  const uint8_t* action_mask, const agrl_options* opt,
                                  void* workspace, size_t ws_bytes, float* logp, float* lse,
                                  void* stream) {
  using namespace agrl;
  Common c;
  int rc = validate("agrl_token_logprob", T, max_act, d, V, dtype, H, W, token_id, action_mask,
                    nullptr, nullptr, 0.0f, 0.0f, 0, opt, workspace, ws_bytes, &c, false);
  if (rc) return rc;
  if (T > 0 && (!logp || !lse)) return fail(AGRL_E_NULL, "agrl_token_logprob: output pointer is NULL");
  if (T == 0) return AGRL_OK;
  c.o.kl_beta = 0.0f;          // loss-only options play no part here
  c.o.token_weight = nullptr;
  hipStream_t s = (hipStream_t)stream;
  int* err = device_error_ptr();
  if (!err) return hip_status(hipErrorInvalidSymbol);
  Layout L;
  make_layout(T, c.max_act, d, V, dtype, c.o, &L);
  uint8_t* ws = (uint8_t*)workspace;
  compact(c, L, ws, action_mask, token_id, nullptr, nullptr, nullptr, nullptr, 0.0f, 0, logp,
          lse, H, err, s);
  if (dtype == AGRL_BF16)
    fwd_gemm<__bf16>(c, L, ws, W, s);
  else
    fwd_gemm<float>(c, L, ws, W, s);
  // the loss merge with zero advantages: lse and logp are formed exactly as in
  // the policy-loss forward; its (zero) surrogate partials are not finalised
  MergeArgs m;
  m.ctrl = (const int32_t*)(ws + L.ctrl);
  m.tiles_v = L.tiles_v;
  m.part = (const f32x2*)(ws + L.part);
  m.ld_part = L.A_pad;
  m.zy = (const float*)(ws + L.zy);
  m.y_act = (const int32_t*)(ws + L.y_act);
  m.old_act = (const float*)(ws + L.old_act);
  m.adv_act = (const float*)(ws + L.adv_act);
  m.idx = (const int32_t*)(ws + L.idx);
  m.eps_lo = 0.0f;
  m.eps_hi = 0.0f;
  m.ref_act = (const float*)(ws + L.ref_act);
  m.w_act = (const float*)(ws + L.w_act);
  m.kl_beta = 0.0f;
  m.kl_est = 0;
  m.weighted = 0;
  m.logp_out = logp;
  m.lse_out = lse;
  m.blk_sum = (double*)(ws + L.blk_sum);
  m.blk_clip = (long long*)(ws + L.blk_clip);
  hipLaunchKernelGGL(merge_loss_kernel, dim3(L.merge_blocks), dim3(256), 0, s, m);
  return hip_status(hipGetLastError());
}

extern "C" int agrl_policy_loss_bwd(int64_t T, int64_t max_act, int32_t d, int32_t V,
                                    int32_t dtype, const void* H, const void* W,
                                    const int32_t* token_id, const uint8_t* action_mask,
                                    const float* adv_tok, const float* old_logp,
                                    float clip_eps_low, float clip_eps_high, int64_t n_norm,
                                    const agrl_options* opt, const float* lse, const float* logp,
                                    float grad_loss, void* workspace, size_t ws_bytes, float* dH,
                                    float* dW, void* stream) {
  using namespace agrl;
  Common c;
  int rc = validate("agrl_policy_loss_bwd", T, max_act, d, V, dtype, H, W, token_id, action_mask,
                    adv_tok, old_logp, clip_eps_low, clip_eps_high, n_norm, opt, workspace,
                    ws_bytes, &c);
  if (rc) return rc;
  if (!dW || (T > 0 && (!dH || !lse || !logp)))
    return fail(AGRL_E_NULL, "agrl_policy_loss_bwd: lse/logp/dH/dW pointer is NULL");
  if (((uintptr_t)dH | (uintptr_t)dW) % 16 != 0)
    return fail(AGRL_E_UNSUPPORTED, "agrl_policy_loss_bwd: dH and dW must be 16-byte aligned");
  if (!isfinite(grad_loss)) return fail(AGRL_E_FLAGS, "agrl_policy_loss_bwd: grad_loss must be finite");
  hipStream_t s = (hipStream_t)stream;
  int* err = device_error_ptr();
  if (!err) return hip_status(hipErrorInvalidSymbol);
  if (T == 0) {
    if (!c.o.dw_accumulate) {
      const int64_t n = (int64_t)V * d;
      hipLaunchKernelGGL(zero_f32_kernel, dim3((unsigned)(n / 256 < 4096 ? n / 256 + 1 : 4096)),
                         dim3(256), 0, s, dW, n);
    }
    return hip_status(hipGetLastError());
  }
  Layout L;
  make_layout(T, c.max_act, d, V, dtype, c.o, &L);
  uint8_t* ws = (uint8_t*)workspace;
  compact(c, L, ws, action_mask, token_id, adv_tok, old_logp, lse, logp, grad_loss, n_norm,
          nullptr, nullptr, H, err, s);
  hipLaunchKernelGGL(zero_masked_rows_kernel, dim3((unsigned)(T < 8192 ? T : 8192)), dim3(256), 0,
                     s, T, d, action_mask, dH);
  if (dtype == AGRL_BF16)
    bwd_gemms<__bf16>(c, L, ws, W, dH, dW, s);
  else
    bwd_gemms<float>(c, L, ws, W, dH, dW, s);
  return hip_status(hipGetLastError());
}
