// a1 router projection and a2 top-k routing.
//
// Top-k: one wave per token. Lane l holds logits of experts l, l+64, ...; k
// rounds of a wave-wide arg-max over (logit descending, id ascending) pick the
// experts in their fixed order (ties to the lower id: paper, Correctness
// recovery / Later numerical and integration repairs). Lanes 0..k-1 keep pick
// j = lane; the renormalised softmax weights are formed from them with the
// denominator summed in pick order.
#include "moe_dev.h"
#include "moe_launch.h"

namespace moe {

// logits[t, e] = sum_h x[t, h] * wr[e, h]; one wave per (t, e). Each lane
// accumulates 8 consecutive h per step (fmaf, fixed order), then a fixed
// butterfly sums the 64 lane partials.
__global__ __launch_bounds__(256) void router_logits_kernel(const uint16_t* __restrict__ x,
                                                            const uint16_t* __restrict__ wr, int T,
                                                            int H, int E,
                                                            float* __restrict__ logits) {
  const long wave = ((long)blockIdx.x * blockDim.x + threadIdx.x) / kWave;
  const int lane = threadIdx.x % kWave;
  if (wave >= (long)T * E) return;
  const int t = (int)(wave / E), e = (int)(wave % E);
  const uint16_t* xr = x + (size_t)t * H;
  const uint16_t* wrow = wr + (size_t)e * H;
  float acc = 0.0f;
  for (int h = lane * 8; h < H; h += kWave * 8) {
    const uint4 xv = *reinterpret_cast<const uint4*>(xr + h);
    const uint4 wv = *reinterpret_cast<const uint4*>(wrow + h);
    const uint32_t xs[4] = {xv.x, xv.y, xv.z, xv.w};
    const uint32_t ws[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc = fmaf(bf16_to_f32(xs[i] & 0xffffu), bf16_to_f32(ws[i] & 0xffffu), acc);
      acc = fmaf(bf16_to_f32(xs[i] >> 16), bf16_to_f32(ws[i] >> 16), acc);
    }
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) acc += shfl_xor_f(acc, m);
  if (lane == 0) logits[(size_t)t * E + e] = acc;
}

// EPL = experts held per lane (ceil(E / 64) rounded up to a power of two).
template <int EPL>
__global__ __launch_bounds__(256) void route_topk_kernel(const float* __restrict__ logits, int T,
                                                         int E, int k, int n_shared,
                                                         int32_t* __restrict__ ids,
                                                         float* __restrict__ wts) {
  const int t = (int)(((long)blockIdx.x * blockDim.x + threadIdx.x) / kWave);
  const int lane = threadIdx.x % kWave;
  if (t >= T) return;
  const float* row = logits + (size_t)t * E;
  float v[EPL];
  bool live[EPL];
#pragma unroll
  for (int j = 0; j < EPL; ++j) {
    const int e = lane + kWave * j;
    live[j] = e < E;
    float x = live[j] ? row[e] : -INFINITY;
    v[j] = (x != x) ? -INFINITY : x;  // NaN reads as -inf
  }
  float my_val = 0.0f;
  int my_id = 0;
  for (int r = 0; r < k; ++r) {
    float bv = -INFINITY;
    int bi = 0x7fffffff;
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const int e = lane + kWave * j;
      if (live[j] && (v[j] > bv || (v[j] == bv && e < bi))) {
        bv = v[j];
        bi = e;
      }
    }
    wave_argmax(bv, bi);
    // every lane now holds the same (bv, bi); retire the pick
#pragma unroll
    for (int j = 0; j < EPL; ++j)
      if (lane + kWave * j == bi) live[j] = false;
    if (lane == r) {
      my_val = bv;
      my_id = bi;
    }
  }
  const float l0 = lane_value(my_val, 0);
  const float ex = lane < k ? expf(my_val - l0) : 0.0f;
  float den = 0.0f;
  for (int j = 0; j < k; ++j) den += lane_value(ex, j);
  const int kt = k + n_shared;
  int32_t* id_row = ids + (size_t)t * kt;
  float* w_row = wts + (size_t)t * kt;
  if (lane < k) {
    id_row[lane] = my_id;
    w_row[lane] = ex / den;
  } else if (lane == k && n_shared) {
    id_row[lane] = E;
    w_row[lane] = 1.0f;
  }
}

// Routing variants. One wave per token, lane l holds experts l, l + 64, ...
// Keys: without a bias the raw logits (every score is increasing in the
// logit); with one, s_e + bias[e] in fp32. Groups: each group's top-two key
// sum is reduced over the wave (lane g keeps group g's score), k rounds of
// arg-max over the lanes pick the kept groups, and their ballot masks the
// experts of the other groups. Then k rounds of arg-max over the keys pick
// the experts, as in route_topk_kernel.
__device__ __forceinline__ void top2_merge(float& a1, float& a2, float b1, float b2) {
  // (a1 >= a2), (b1 >= b2): the two largest of the four
  const float hi = fmaxf(a1, b1);
  const float lo = a1 >= b1 ? fmaxf(a2, b1) : fmaxf(a1, b2);
  a1 = hi;
  a2 = lo;
}

// Routing of one token whose E logits are at `row` (global or LDS), by the
// calling wave; writes its k + n_shared ids and weights.
template <int EPL>
__device__ __forceinline__ void route_token(const float* row, int E, int k, int n_shared,
                                            const RouteOpts& o, int32_t* id_row, float* w_row,
                                            int lane) {
  float l[EPL], key[EPL];
  bool live[EPL];
  float lmax = -INFINITY;
#pragma unroll
  for (int j = 0; j < EPL; ++j) {
    const int e = lane + kWave * j;
    live[j] = e < E;
    const float x = live[j] ? row[e] : -INFINITY;
    l[j] = (x != x) ? -INFINITY : x;  // NaN reads as -inf
    lmax = fmaxf(lmax, l[j]);
  }
  static_for<6>([&](auto L) {
    lmax = fmaxf(lmax, __int_as_float(wave_partner<decltype(L)::value>(__float_as_int(lmax))));
  });
  // softmax denominator, summed in a fixed order (lane order j, then butterfly)
  float den = 0.0f;
  if (!o.sigmoid) {
#pragma unroll
    for (int j = 0; j < EPL; ++j)
      if (live[j]) den += expf(l[j] - lmax);
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) den += shfl_xor_f(den, m);
  }
  auto score = [&](float x) {
    return o.sigmoid ? 1.0f / (1.0f + expf(-x)) : expf(x - lmax) / den;
  };
#pragma unroll
  for (int j = 0; j < EPL; ++j) {
    const int e = lane + kWave * j;
    key[j] = !live[j] ? -INFINITY : (o.bias ? score(l[j]) + o.bias[e] : l[j]);
  }
  if (o.n_group > 1) {
    const int gs = E / o.n_group;
    float my_gs = -INFINITY;
    for (int g = 0; g < o.n_group; ++g) {
      float a1 = -INFINITY, a2 = -INFINITY;
#pragma unroll
      for (int j = 0; j < EPL; ++j) {
        const int e = lane + kWave * j;
        if (live[j] && e / gs == g) {
          // group scores always use the fp32 key value s + bias
          const float v = o.bias ? key[j] : score(l[j]);
          top2_merge(a1, a2, v, -INFINITY);
        }
      }
      static_for<6>([&](auto L) {  // the two largest over the wave (a multiset union)
        constexpr int l = decltype(L)::value;
        const float b1 = __int_as_float(wave_partner<l>(__float_as_int(a1)));
        const float b2 = __int_as_float(wave_partner<l>(__float_as_int(a2)));
        top2_merge(a1, a2, b1, b2);
      });
      if (lane == g) my_gs = gs == 1 ? a1 : a1 + a2;
    }
    // keep topk_group groups: arg-max rounds over (score descending, group ascending)
    bool kept = false;
    for (int r = 0; r < o.topk_group; ++r) {
      float bv = (lane < o.n_group && !kept) ? my_gs : -INFINITY;
      int bi = (lane < o.n_group && !kept) ? lane : 0x7fffffff;
      wave_argmax(bv, bi);
      if (lane == bi) kept = true;
    }
    const uint64_t mask = __ballot(kept);
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const int e = lane + kWave * j;
      if (live[j] && !((mask >> (e / gs)) & 1)) live[j] = false;
    }
  }
  float my_key = 0.0f, my_l = 0.0f;
  int my_id = 0;
  for (int r = 0; r < k; ++r) {
    float bv = -INFINITY, bl = 0.0f;
    int bi = 0x7fffffff;
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const int e = lane + kWave * j;
      if (live[j] && (key[j] > bv || (key[j] == bv && e < bi))) {
        bv = key[j];
        bi = e;
        bl = l[j];
      }
    }
    static_for<6>([&](auto L) {  // arg-max carrying the pick's logit
      constexpr int q = decltype(L)::value;
      const float ov = __int_as_float(wave_partner<q>(__float_as_int(bv)));
      const float ol = __int_as_float(wave_partner<q>(__float_as_int(bl)));
      const int oi = wave_partner<q>(bi);
      if (ov > bv || (ov == bv && oi < bi)) {
        bv = ov;
        bi = oi;
        bl = ol;
      }
    });
#pragma unroll
    for (int j = 0; j < EPL; ++j)
      if (lane + kWave * j == bi) live[j] = false;
    if (lane == r) {
      my_key = bv;
      my_id = bi;
      my_l = bl;
    }
  }
  (void)my_key;
  float wv;
  if (!o.sigmoid && o.renorm) {
    // exactly moe_route_topk's weights: exp(l_j - l_0) / sum over the picks
    const float l0 = lane_value(my_l, 0);
    wv = lane < k ? expf(my_l - l0) : 0.0f;
  } else {
    wv = lane < k ? score(my_l) : 0.0f;
  }
  if (o.renorm) {
    float sum = 0.0f;
    for (int j = 0; j < k; ++j) sum += lane_value(wv, j);
    wv = wv / sum;
  }
  wv *= o.scale;
  if (lane < k) {
    id_row[lane] = my_id;
    w_row[lane] = wv;
  } else if (lane == k && n_shared) {
    id_row[lane] = E;
    w_row[lane] = 1.0f;
  }
}

template <int EPL>
__global__ __launch_bounds__(256) void route_topk_ex_kernel(const float* __restrict__ logits, int T,
                                                            int E, int k, int n_shared,
                                                            RouteOpts o,
                                                            int32_t* __restrict__ ids,
                                                            float* __restrict__ wts) {
  const int t = (int)(((long)blockIdx.x * blockDim.x + threadIdx.x) / kWave);
  const int lane = threadIdx.x % kWave;
  if (t >= T) return;
  const int kt = k + n_shared;
  route_token<EPL>(logits + (size_t)t * E, E, k, n_shared, o, ids + (size_t)t * kt,
                   wts + (size_t)t * kt, lane);
}

// Fused router projection and routing (f1). A workgroup owns 32 tokens and
// all E experts, in chunks of 256: wave w computes logits of experts
// [c0 + 64 w, +64) of chunk c0 for the 32 tokens on the 32x32x16 bf16 matrix
// cores (products exact, fp32 accumulation), operands loaded straight to
// registers (row l % 32 and 8 consecutive K elements per lane, the same
// placement for both operands); the 32 x E logits go to LDS (row stride
// rt_stride(E), odd), then each wave routes 8 of the tokens.
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef float v16f_r __attribute__((ext_vector_type(16)));

constexpr int kRtTok = 32;  // tokens per workgroup

// fp32 row stride of the LDS logits: E rounded up to 64, plus one.
__host__ __device__ inline int rt_stride(int E) { return (E + 63) / 64 * 64 + 1; }

template <int EPL>
__global__ __launch_bounds__(256) void router_topk_kernel(const uint16_t* __restrict__ x,
                                                          const uint16_t* __restrict__ wr, int T,
                                                          int H, int E, int k, int n_shared,
                                                          RouteOpts o, float* __restrict__ logits,
                                                          int32_t* __restrict__ ids,
                                                          float* __restrict__ wts) {
  extern __shared__ float lg[];  // [kRtTok][stride]
  const int stride = rt_stride(E);
  const int t0 = blockIdx.x * kRtTok;
  const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int r = lane & 31, h = lane >> 5;
  const int ng = H / 128;  // groups of 128 K elements
  if (ng * 128 != H) return;  // the launcher only passes H % 128 == 0
  // operand rows (clamped to valid rows; the extra results are never used)
  const uint16_t* xa = x + (size_t)min(t0 + r, T - 1) * H + 8 * h;
  for (int c0 = 0; c0 < E; c0 += 256) {
    const int e0 = c0 + 64 * w;  // this wave's first expert of the chunk
    const uint16_t* wb0 = wr + (size_t)min(e0 + r, E - 1) * H + 8 * h;
    const uint16_t* wb1 = wr + (size_t)min(e0 + 32 + r, E - 1) * H + 8 * h;
    v16f_r acc0 = v16f_r{}, acc1 = v16f_r{};
    constexpr int kU = 8;  // K steps of 16 per group (two groups of loads in flight)
    v8bf a[2][kU], b0[2][kU], b1[2][kU];
    auto load = [&](int buf, int k0) {
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int kk = k0 + 16 * u;
        a[buf][u] = *reinterpret_cast<const v8bf*>(xa + kk);
        b0[buf][u] = *reinterpret_cast<const v8bf*>(wb0 + kk);
        b1[buf][u] = *reinterpret_cast<const v8bf*>(wb1 + kk);
      }
    };
    auto mma = [&](int buf) {
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[buf][u], b0[buf][u], acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[buf][u], b1[buf][u], acc1, 0, 0, 0);
      }
    };
    load(0, 0);
    int g = 0;
    for (; g + 2 <= ng; g += 2) {
      if (g + 1 < ng) load(1, 16 * kU * (g + 1));
      mma(0);
      if (g + 2 < ng) load(0, 16 * kU * (g + 2));
      mma(1);
    }
    if (g < ng) mma(0);
    // D: lane l, element i = token 8 (i / 4) + 4 h + i % 4, expert column l % 32
    // (columns at or past E are padding: stored, never read)
    if (e0 < E) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int tr = 8 * (i / 4) + 4 * h + (i % 4);
        lg[tr * stride + e0 + r] = acc0[i];
        lg[tr * stride + e0 + 32 + r] = acc1[i];
      }
    }
  }
  __syncthreads();
  const int kt = k + n_shared;
  for (int tt = w; tt < kRtTok; tt += 4) {
    const int t = t0 + tt;
    if (t >= T) break;
    const float* row = lg + tt * stride;
    if (logits)
      for (int e = lane; e < E; e += kWave) logits[(size_t)t * E + e] = row[e];
    route_token<EPL>(row, E, k, n_shared, o, ids + (size_t)t * kt, wts + (size_t)t * kt, lane);
  }
}

hipError_t launch_router_topk(const uint16_t* x, const uint16_t* wr, int T, int H, int E, int k,
                              int n_shared, const RouteOpts& o, float* logits, int32_t* ids,
                              float* w, hipStream_t s) {
  if (T == 0) return hipSuccess;
  const int blocks = (T + kRtTok - 1) / kRtTok;
  const int epl = (E + kWave - 1) / kWave;
  const size_t lds = (size_t)kRtTok * rt_stride(E) * sizeof(float);
#define MOE_RT(N)                                                                               \
  hipLaunchKernelGGL(router_topk_kernel<N>, dim3(blocks), dim3(256), lds, s, x, wr, T, H, E, k, \
                     n_shared, o, logits, ids, w)
  if (epl <= 1)
    MOE_RT(1);
  else if (epl <= 2)
    MOE_RT(2);
  else if (epl <= 4)
    MOE_RT(4);
  else if (epl <= 8)
    MOE_RT(8);
  else
    MOE_RT(16);
#undef MOE_RT
  return hipGetLastError();
}

hipError_t launch_route_topk_ex(const float* logits, int T, int E, int k, int n_shared,
                                const RouteOpts& o, int32_t* ids, float* w, hipStream_t s) {
  if (T == 0) return hipSuccess;
  const int blocks = (T + 3) / 4;
  const int epl = (E + kWave - 1) / kWave;
#define MOE_ROUTE_EX(N)                                                                       \
  hipLaunchKernelGGL(route_topk_ex_kernel<N>, dim3(blocks), dim3(256), 0, s, logits, T, E, k, \
                     n_shared, o, ids, w)
  if (epl <= 1)
    MOE_ROUTE_EX(1);
  else if (epl <= 2)
    MOE_ROUTE_EX(2);
  else if (epl <= 4)
    MOE_ROUTE_EX(4);
  else if (epl <= 8)
    MOE_ROUTE_EX(8);
  else
    MOE_ROUTE_EX(16);
#undef MOE_ROUTE_EX
  return hipGetLastError();
}

hipError_t launch_router_logits(const uint16_t* x, const uint16_t* wr, int T, int H, int E,
                                float* logits, hipStream_t s) {
  const long waves = (long)T * E;
  if (waves == 0) return hipSuccess;
  const int blocks = (int)((waves * kWave + 255) / 256);
  hipLaunchKernelGGL(router_logits_kernel, dim3(blocks), dim3(256), 0, s, x, wr, T, H, E, logits);
  return hipGetLastError();
}

hipError_t launch_route_topk(const float* logits, int T, int E, int k, int n_shared, int32_t* ids,
                             float* w, hipStream_t s) {
  if (T == 0) return hipSuccess;
  const int blocks = (T + 3) / 4;  // 4 waves (tokens) per 256-thread block
  const int epl = (E + kWave - 1) / kWave;
#define MOE_ROUTE(N)                                                                      \
  hipLaunchKernelGGL(route_topk_kernel<N>, dim3(blocks), dim3(256), 0, s, logits, T, E, k, \
                     n_shared, ids, w)
  if (epl <= 1)
    MOE_ROUTE(1);
  else if (epl <= 2)
    MOE_ROUTE(2);
  else if (epl <= 4)
    MOE_ROUTE(4);
  else if (epl <= 8)
    MOE_ROUTE(8);
  else
    MOE_ROUTE(16);
#undef MOE_ROUTE
  return hipGetLastError();
}

}  // namespace moe
