// Router logits z_t = W_r h_t (Sec. 3.1): an fp32 [T,H] x [E,H]^T product on
// the fp32 MFMA (v_mfma_f32_16x16x4f32), one 16-token x 16-expert tile per
// workgroup of 16 waves.  Each wave reduces a contiguous slice of H; the
// loads of a batch of 8 chunks are all issued before its first MFMA, so a
// wave waits for memory once per batch rather than once per chunk (rows past
// T / E are clamped, computed and dropped).  The 16 partial tiles are summed
// in LDS in a fixed order (deterministic).
#include "common.hpp"
#include "launch.hpp"

namespace amoe {

namespace {

constexpr int kRouteWaves = 16;
constexpr int kRouteBatch = 8;  // 16-wide K chunks loaded ahead of their MFMAs

// Raw loads of four consecutive inputs, widened to fp32 only after the whole
// batch has been issued (widening right after each load would make the wave
// wait for it before issuing the next).
__device__ __forceinline__ float4 load_raw(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ uint2 load_raw(const uint16_t* p) { return *reinterpret_cast<const uint2*>(p); }

__device__ __forceinline__ float4 widen(const float4& v) { return v; }
__device__ __forceinline__ float4 widen(const uint2& v) {
  return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
                     __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u));
}

template <typename TIn>
struct Raw4 {
  typedef float4 type;
};
template <>
struct Raw4<uint16_t> {
  typedef uint2 type;
};

// grid (ceil(E/16), ceil(T/16)), block 1024.  Lane (r, g): token row t0 + r of
// the A tile and expert column e0 + r of the B tile; K slice g of each
// 16-wide chunk is the float4 at offset 4g, component j feeds MFMA j.
template <typename TIn>
__global__ __launch_bounds__(kRouteWaves * kWave) void route_kernel(const TIn* __restrict__ hidden,
                                                                   const float* __restrict__ w, int T, int H,
                                                                   int E, float* __restrict__ logits) {
  __shared__ floatx4 part[kRouteWaves][kWave];
  const int wave = wave_id();
  const int lane = lane_id();
  const int r = lane & 15, g = lane >> 4;
  const int e0 = blockIdx.x * 16, t0 = blockIdx.y * 16;
  const int t = min(t0 + r, T - 1), e = min(e0 + r, E - 1);
  const TIn* hrow = hidden + static_cast<size_t>(t) * H + 4 * g;
  const float* wrow = w + static_cast<size_t>(e) * H + 4 * g;

  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
  const int nchunk = H / 16;
  const int c0 = wave * nchunk / kRouteWaves, c1 = (wave + 1) * nchunk / kRouteWaves;
  for (int cb = c0; cb < c1; cb += kRouteBatch) {
    // chunks past c1 re-read chunk c1 - 1 and are not used
    typename Raw4<TIn>::type ar[kRouteBatch];
    float4 b[kRouteBatch];
#pragma unroll
    for (int i = 0; i < kRouteBatch; ++i) {
      const int c = min(cb + i, c1 - 1);
      ar[i] = load_raw(hrow + c * 16);
      b[i] = load_raw(wrow + c * 16);
    }
    // keep the scheduler from sinking each load down to its MFMA
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < kRouteBatch; ++i) {
      const float4 a = widen(ar[i]);
      floatx4 n = mfma_f32_16x16x4(a.x, b[i].x, acc);
      n = mfma_f32_16x16x4(a.y, b[i].y, n);
      n = mfma_f32_16x16x4(a.z, b[i].z, n);
      n = mfma_f32_16x16x4(a.w, b[i].w, n);
      acc = cb + i < c1 ? n : acc;  // wave-uniform select, no branch
    }
  }
  part[wave][lane] = acc;
  __syncthreads();
  if (wave == 0) {
    floatx4 s = part[0][lane];
#pragma unroll
    for (int w2 = 1; w2 < kRouteWaves; ++w2) {
      const floatx4 q = part[w2][lane];
      s[0] += q[0];
      s[1] += q[1];
      s[2] += q[2];
      s[3] += q[3];
    }
    if (e0 + r < E) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int tt = t0 + 4 * g + i;
        if (tt < T) logits[static_cast<size_t>(tt) * E + e0 + r] = s[i];
      }
    }
  }
}

}  // namespace

hipError_t launch_route(const void* hidden, int hidden_is_bf16, const float* router_w, int T, int H,
                        int E, float* logits, hipStream_t stream) {
  dim3 grid((E + 15) / 16, (T + 15) / 16);
  const int block = kRouteWaves * kWave;
  if (hidden_is_bf16)
    route_kernel<uint16_t><<<grid, block, 0, stream>>>(static_cast<const uint16_t*>(hidden), router_w, T, H,
                                                       E, logits);
  else
    route_kernel<float><<<grid, block, 0, stream>>>(static_cast<const float*>(hidden), router_w, T, H, E,
                                                    logits);
  return hipGetLastError();
}

}  // namespace amoe
