// Inference of the draft policies (section 4: state vector; appendix A.2:
// fully connected ReLU networks, hidden [1024, 256] for the size policy and
// [1024] for the depth policy, argmax action).
//
// A batch of B states is tiny next to the weights (4 MB for the size policy's
// first layer), so every layer is a weight-streaming GEMV over at most eight
// states at a time:
//
//   dense_kernel   one output unit per wave, four per workgroup: each lane
//                  holds its stride-64 share of the unit's weight row in
//                  registers (loaded first), the layer's input for up to
//                  eight states (the batch rounded up to a power of two; more
//                  states take more workgroups) sits in LDS transposed (k-major, rows
//                  padded against bank conflicts), each lane keeps one
//                  partial sum per state, and a butterfly over the lanes
//                  reduces them with permlane swaps and DPP moves (halving
//                  exchanges while there are several sums, plain ones after).
//                  The first layer builds its input straight from the draft
//                  pool's scores (no separate state pass).  Every load is
//                  unconditional, clamped in bounds, and issued before the
//                  first wait;
//   head_kernel    one workgroup per state: the output logits (one wave per
//                  logit, lanes over the hidden units), then the argmax
//                  (lowest index on ties) mapped to offset + scale * index.
//
// Weights are float32, [out][in] row-major; accumulation is float32 in a
// fixed order (deterministic).  The layers are HBM/L2-latency bound, not ALU
// bound: B*in*out FMAs (16.6M for B = 16 on the first layer) take under a
// microsecond spread over the chip.
#include "ltd_device.hpp"
#include "ltd_launch.hpp"

namespace ltd {
namespace {

constexpr int kThreads = 256;
constexpr int kUnitsPerBlock = kThreads / kWave;
constexpr int kMaxStates = 8;  // states per LDS chunk (= partial sums per lane)
constexpr int kStageSteps = LTD_POLICY_MAX_IN / kThreads;
constexpr int kRowSteps = LTD_POLICY_MAX_IN / kWave;
constexpr int kHeadSteps = LTD_POLICY_MAX_HIDDEN / kWave;
static_assert(LTD_POLICY_MAX_IN % kThreads == 0 && LTD_POLICY_MAX_HIDDEN % kWave == 0, "");
// LDS row stride of the staged inputs: padded past four states so that the
// lanes' 16-byte reads of consecutive rows hit distinct banks
template <int kStates>
constexpr int stage_stride() {
  return kStates <= 4 ? kStates : kStates + 4;
}
static_assert(LTD_POLICY_MAX_IN * stage_stride<kMaxStates>() * 4 <= 65536, "staged inputs fit LDS");

struct PoolInput {
  const float* scores;
  const int32_t* pool_size;
  const int32_t* depth;
  const int32_t* ctx_len;
  int Vpool;
  int layout;
  float pad;
};

// One halving level of the butterfly at distance `dist`: lanes with that bit
// set keep the upper half of the partial sums, the others the lower half, and
// each adds its partner's copy of what it keeps.
template <int kHalf, int kDist>
__device__ __forceinline__ void halve(float* acc, int lane) {
  const bool upper = lane & kDist;
#pragma unroll
  for (int q = 0; q < kHalf; ++q) {
    float from_partner;
    if constexpr (kDist >= 16) {
      const unsigned a = __float_as_uint(acc[q]);
      const unsigned b = __float_as_uint(acc[q + kHalf]);
      if constexpr (kDist == 32) {
        const auto r = __builtin_amdgcn_permlane32_swap(a, b, false, false);
        from_partner = __uint_as_float(upper ? r[0] : r[1]);
      } else {
        const auto r = __builtin_amdgcn_permlane16_swap(a, b, false, false);
        from_partner = __uint_as_float(upper ? r[0] : r[1]);
      }
    } else {
      from_partner = lane_xor_f<kDist>(upper ? acc[q] : acc[q + kHalf], lane);
    }
    acc[q] = (upper ? acc[q + kHalf] : acc[q]) + from_partner;
  }
}

// Sum of v over all 64 lanes, in every lane.
__device__ __forceinline__ float wave_total(float v, int lane) {
  v += lane_xor_f<32>(v, lane);
  v += lane_xor_f<16>(v, lane);
  v += lane_xor_f<8>(v, lane);
  v += lane_xor_f<4>(v, lane);
  v += lane_xor_f<2>(v, lane);
  v += lane_xor_f<1>(v, lane);
  return v;
}

// Where a layer's input comes from.
enum Source { kHidden = 0, kPoolSize = 1, kPoolDepth = 2 };

// One output unit per wave, four per workgroup; kStates states per
// workgroup, blockIdx.y picks the chunk of states.
template <int kStates, int kSource>
__global__ void __launch_bounds__(kThreads) dense_kernel(const float* __restrict__ x, PoolInput pool,
                                                         int B, int in_dim,
                                                         const float* __restrict__ w,
                                                         const float* __restrict__ bias,
                                                         int out_dim, float* __restrict__ y) {
  static_assert(kStates >= 1 && kStates <= kMaxStates && (kStates & (kStates - 1)) == 0, "");
  constexpr int kLevels = kStates == 1 ? 0 : kStates == 2 ? 1 : kStates == 4 ? 2 : kStates == 8 ? 3 : 4;
  constexpr int kStride = stage_stride<kStates>();
  __shared__ float x_s[LTD_POLICY_MAX_IN * kStride];  // k-major: x_s[k * kStride + s]
  const int lane = threadIdx.x & (kWave - 1);
  const int unit = blockIdx.x * kUnitsPerBlock + threadIdx.x / kWave;
  const bool active = unit < out_dim;
  const float* wrow = w + static_cast<int64_t>(min(unit, out_dim - 1)) * in_dim;

  // the unit's weight row (zeros past in_dim), requested before anything else
  float wreg[kRowSteps];
#pragma unroll
  for (int i = 0; i < kRowSteps; ++i) {
    const int k = lane + i * kWave;
    const float v = wrow[min(k, in_dim - 1)];
    wreg[i] = k < in_dim ? v : 0.f;
  }
  const float bj = bias[min(unit, out_dim - 1)];
  const int n_feat = in_dim - 2;

  constexpr bool kFromPool = kSource != kHidden;
  {
    const int b0 = blockIdx.y * kStates;
    // stage the inputs of states b0 .. b0+kStates-1, k-major, zeros past B and
    // past in_dim.  The per-state scalars arrive with one vector load each
    // (lane s holds state s's) and are broadcast with readlane; every other
    // load is unconditional (clamped in bounds) and issued before any wait.
    int n_lane = 0, d_lane = 0, l_lane = 0;
    if constexpr (kFromPool) {
      const int bl = min(b0 + (lane & (kStates - 1)), B - 1);
      n_lane = min(max(pool.pool_size[bl], 0), pool.Vpool);
      d_lane = pool.depth[bl];
      l_lane = pool.ctx_len[bl];
    }
    float v[kStates][kStageSteps];
#pragma unroll
    for (int s = 0; s < kStates; ++s) {
      const int b = min(b0 + s, B - 1);
      if constexpr (kFromPool) {
        const float* row = pool.scores + static_cast<int64_t>(b) * pool.Vpool;
        // the size layout's scores do not depend on the pool size
        const int base = kSource == kPoolSize ? -2 : __builtin_amdgcn_readlane(n_lane, s) - n_feat;
#pragma unroll
        for (int i = 0; i < kStageSteps; ++i) {
          const int k = threadIdx.x + i * kThreads;
          v[s][i] = row[min(max(base + k, 0), pool.Vpool - 1)];
        }
      } else {
#pragma unroll
        for (int i = 0; i < kStageSteps; ++i) {
          const int k = threadIdx.x + i * kThreads;
          v[s][i] = x[static_cast<int64_t>(b) * in_dim + min(k, in_dim - 1)];
        }
      }
    }
#pragma unroll
    for (int s = 0; s < kStates; ++s) {
      const bool live = b0 + s < B;
      int n = 0;
      float dval = 0.f, lval = 0.f;
      if constexpr (kFromPool) {
        n = __builtin_amdgcn_readlane(n_lane, s);
        dval = static_cast<float>(__builtin_amdgcn_readlane(d_lane, s));
        lval = static_cast<float>(__builtin_amdgcn_readlane(l_lane, s));
      }
#pragma unroll
      for (int i = 0; i < kStageSteps; ++i) {
        const int k = threadIdx.x + i * kThreads;
        float e = v[s][i];
        if constexpr (kFromPool) {
          constexpr bool size = kSource == kPoolSize;
          const int kd = size ? 0 : n_feat;  // position of D; L follows it
          const bool padded = size ? k - 2 >= min(n, n_feat) : n - n_feat + k < 0;
          e = padded ? pool.pad : e;
          e = k == kd ? dval : e;
          e = k == kd + 1 ? lval : e;
        }
        x_s[k * kStride + s] = live && k < in_dim ? e : 0.f;
      }
    }
    __syncthreads();

    float acc[kStates];
#pragma unroll
    for (int s = 0; s < kStates; ++s) acc[s] = 0.f;
#pragma unroll
    for (int i = 0; i < kRowSteps; ++i) {
      const int k = lane + i * kWave;
      const float wk = wreg[i];
      if constexpr (kStates >= 4) {
#pragma unroll
        for (int q = 0; q < kStates / 4; ++q) {
          const float4 xv = reinterpret_cast<const float4*>(x_s + k * kStride)[q];
          acc[4 * q + 0] = fmaf(wk, xv.x, acc[4 * q + 0]);
          acc[4 * q + 1] = fmaf(wk, xv.y, acc[4 * q + 1]);
          acc[4 * q + 2] = fmaf(wk, xv.z, acc[4 * q + 2]);
          acc[4 * q + 3] = fmaf(wk, xv.w, acc[4 * q + 3]);
        }
      } else {
#pragma unroll
        for (int s = 0; s < kStates; ++s) acc[s] = fmaf(wk, x_s[k * kStride + s], acc[s]);
      }
    }
    // butterfly over the lanes: kLevels halving levels at distances 32, 16,
    // ... then plain sums at the remaining distances; lane l ends with the
    // sum for state l >> (6 - kLevels), shared by its group of lanes
    if constexpr (kLevels >= 1) halve<kStates / 2, 32>(acc, lane);
    if constexpr (kLevels >= 2) halve<kStates / 4, 16>(acc, lane);
    if constexpr (kLevels >= 3) halve<kStates / 8, 8>(acc, lane);
    if constexpr (kLevels >= 4) halve<kStates / 16, 4>(acc, lane);
    float r = acc[0];
    if constexpr (kLevels < 1) r += lane_xor_f<32>(r, lane);
    if constexpr (kLevels < 2) r += lane_xor_f<16>(r, lane);
    if constexpr (kLevels < 3) r += lane_xor_f<8>(r, lane);
    if constexpr (kLevels < 4) r += lane_xor_f<4>(r, lane);
    r += lane_xor_f<2>(r, lane);
    r += lane_xor_f<1>(r, lane);
    constexpr int kGroupBits = 6 - kLevels;
    const int b = b0 + (lane >> kGroupBits);
    if (active && (lane & ((1 << kGroupBits) - 1)) == 0 && b < B)
      y[static_cast<int64_t>(b) * out_dim + unit] = fmaxf(r + bj, 0.f);  // ReLU
  }
}

__global__ void __launch_bounds__(kThreads) head_kernel(const float* __restrict__ h, int hidden,
                                                        const float* __restrict__ w,
                                                        const float* __restrict__ bias, int n_out,
                                                        int action_offset, int action_scale,
                                                        float* __restrict__ logits,
                                                        int32_t* __restrict__ action) {
  __shared__ float logit_s[LTD_POLICY_MAX_OUT];
  const int b = blockIdx.x;
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = threadIdx.x / kWave;
  // this lane's share of the state's hidden activations (zeros past hidden)
  float hreg[kHeadSteps];
#pragma unroll
  for (int i = 0; i < kHeadSteps; ++i) {
    const int k = lane + i * kWave;
    const float v = h[static_cast<int64_t>(b) * hidden + min(k, hidden - 1)];
    hreg[i] = k < hidden ? v : 0.f;
  }
  for (int o = wv; o < n_out; o += kUnitsPerBlock) {
    const float* wrow = w + static_cast<int64_t>(o) * hidden;
    float wv_[kHeadSteps];
#pragma unroll
    for (int i = 0; i < kHeadSteps; ++i) wv_[i] = wrow[min(lane + i * kWave, hidden - 1)];
    float acc = 0.f;
#pragma unroll
    for (int i = 0; i < kHeadSteps; ++i) acc = fmaf(wv_[i], hreg[i], acc);
    acc = wave_total(acc, lane);
    if (lane == 0) {
      const float v = acc + bias[o];
      logit_s[o] = v;
      logits[static_cast<int64_t>(b) * n_out + o] = v;
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int best = 0;
    for (int o = 1; o < n_out; ++o)
      if (logit_s[o] > logit_s[best]) best = o;
    action[b] = action_offset + action_scale * best;
  }
}

template <int kSource>
void launch_dense(int states, int units, hipStream_t stream, const float* x,
                  const PoolInput& pool, int B, int in_dim, const float* w, const float* bias,
                  int out_dim, float* y) {
  const dim3 grid((units + kUnitsPerBlock - 1) / kUnitsPerBlock, (B + states - 1) / states);
  const dim3 block(kThreads);
  switch (states) {
    case 1:
      hipLaunchKernelGGL((dense_kernel<1, kSource>), grid, block, 0, stream, x, pool, B, in_dim, w,
                         bias, out_dim, y);
      break;
    case 2:
      hipLaunchKernelGGL((dense_kernel<2, kSource>), grid, block, 0, stream, x, pool, B, in_dim, w,
                         bias, out_dim, y);
      break;
    case 4:
      hipLaunchKernelGGL((dense_kernel<4, kSource>), grid, block, 0, stream, x, pool, B, in_dim, w,
                         bias, out_dim, y);
      break;
    default:
      hipLaunchKernelGGL((dense_kernel<8, kSource>), grid, block, 0, stream, x, pool, B, in_dim, w,
                         bias, out_dim, y);
  }
}

}  // namespace

size_t policy_workspace_bytes(int B, int h1, int h2) {
  return sizeof(float) * static_cast<size_t>(B) * (static_cast<size_t>(h1) + h2);
}

hipError_t launch_policy(int layout, const float* scores, const int32_t* pool_size, int Vpool,
                         const int32_t* depth, const int32_t* ctx_len, float pad, int B,
                         int in_dim, const float* w1, const float* b1, int h1, const float* w2,
                         const float* b2, int h2, const float* wo, const float* bo, int n_out,
                         int action_offset, int action_scale, float* logits, int32_t* action,
                         void* workspace, hipStream_t stream) {
  float* a1 = static_cast<float*>(workspace);
  float* a2 = a1 + static_cast<size_t>(B) * h1;
  const PoolInput pool{scores, pool_size, depth, ctx_len, Vpool, layout, pad};
  int states = 1;  // per workgroup; further chunks go to more workgroups
  while (states < B && states < kMaxStates) states <<= 1;
  if (layout == LTD_POLICY_SIZE)
    launch_dense<kPoolSize>(states, h1, stream, nullptr, pool, B, in_dim, w1, b1, h1, a1);
  else
    launch_dense<kPoolDepth>(states, h1, stream, nullptr, pool, B, in_dim, w1, b1, h1, a1);
  const float* last = a1;
  int last_dim = h1;
  if (h2 > 0) {
    launch_dense<kHidden>(states, h2, stream, a1, pool, B, h1, w2, b2, h2, a2);
    last = a2;
    last_dim = h2;
  }
  hipLaunchKernelGGL(head_kernel, dim3(B), dim3(kThreads), 0, stream, last, last_dim, wo, bo,
                     n_out, action_offset, action_scale, logits, action);
  return hipGetLastError();
}

}  // namespace ltd
