// Router logits z_t = W_r h_t (Sec. 3.1): an fp32 [T,H] x [E,H]^T product on
// the fp32 MFMA (v_mfma_f32_16x16x4f32), one 16-token x 16-expert tile (or
// 16 x 8 for small grids) per workgroup of 16 waves, each wave reducing a
// slice of H.
//
// Both operands are read with whole-cache-line accesses: the router weights
// come pre-packed in MFMA fragment order (one contiguous 1 KiB read per
// 16-expert x 16-column chunk, see acceptmoe_pack_router_weights), and the
// workgroup's 16 hidden rows are staged in LDS with row-contiguous loads
// before the waves read their A fragments from there.  A wave issues all of
// its weight loads for a staged block before waiting for the staging, so the
// two transfers overlap.  The 16 partial tiles are summed in LDS in a fixed
// order (deterministic).
#include "common.hpp"
#include "launch.hpp"

namespace amoe {

namespace {

constexpr int kRouteWaves = 16;
constexpr int kRouteThreads = kRouteWaves * kWave;
constexpr int kRouteStageBytes = 64 * 1024;  // hidden bytes staged per block (16 rows)
constexpr int kRouteBatch = 8;               // 16-wide K chunks per wave and staged block
constexpr int kRouteRowPad = 16;             // bytes appended to each staged row (LDS banks)

// Router weights packed like an fp32 expert stack with N = E rows padded to a
// multiple of 16 with zeros: fragment (expert tile et, chunk c) holds, for
// lane L = r + 16 g, the floats 4g .. 4g+3 of columns 16c .. 16c+15 of row
// 16 et + r.
__global__ void pack_router_kernel(const float4* __restrict__ src, float4* __restrict__ dst, int E, int H) {
  const int nchunk = H / 16;
  const size_t total = static_cast<size_t>((E + 15) / 16) * nchunk * kWave;
  for (size_t q = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; q < total;
       q += static_cast<size_t>(gridDim.x) * blockDim.x) {
    const int lane = static_cast<int>(q & 63);
    const size_t f = q >> 6;
    const int c = static_cast<int>(f % nchunk);
    const int et = static_cast<int>(f / nchunk);
    const int row = et * 16 + (lane & 15);
    dst[q] = row < E ? src[(static_cast<size_t>(row) * H + c * 16 + 4 * (lane >> 4)) / 4]
                     : make_float4(0.f, 0.f, 0.f, 0.f);
  }
}

__device__ __forceinline__ float4 widen4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ float4 widen4(const uint16_t* p) {
  const uint2 v = *reinterpret_cast<const uint2*>(p);
  return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
                     __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u));
}

// grid (ceil(E/EW), ceil(T/16)), block 1024, EW = 16 or 8 experts per
// workgroup.  Lane (r, g) of a wave: token row t0 + r of the A tile and expert
// row r of the B tile; component j of K slice g of chunk c is column
// 16c + 4g + j (same for both operands).  With EW = 8 a workgroup reads one
// half of each 16-row weight fragment (rows 0-7 or 8-15: four whole 128-byte
// lines of the 1 KiB fragment), lanes r >= 8 repeat lanes r - 8 and their
// output columns are dropped; twice the workgroups then share the weights,
// which matters when only a few tiles exist (the per-CU read rate bounds a
// small grid).
template <typename TIn, int EW>
__global__ __launch_bounds__(kRouteThreads) void route_kernel(const TIn* __restrict__ hidden,
                                                             const float4* __restrict__ wp, int T, int H, int E,
                                                             float* __restrict__ logits) {
  constexpr int kEb = sizeof(TIn);
  constexpr int kBlockCols = kRouteStageBytes / (16 * kEb);  // staged columns per block
  constexpr int kRowBytes = kBlockCols * kEb + kRouteRowPad;
  static_assert(kBlockCols / 16 <= kRouteWaves * kRouteBatch, "a staged block must fit the wave batches");
  __shared__ __align__(16) unsigned char hs[16 * kRowBytes];
  __shared__ floatx4 part[kRouteWaves][kWave];
  const int tid = threadIdx.x;
  const int wave = wave_id();
  const int lane = lane_id();
  const int r = lane & 15, g = lane >> 4;
  const int e0 = blockIdx.x * EW, t0 = blockIdx.y * 16;
  const int nchunk = H / 16;
  // fragment lane holding expert row (e0 % 16) + (r % EW) for K slice g
  const int wl = (e0 % 16) + (r % EW) + 16 * g;
  const float4* wrow = wp + static_cast<size_t>(e0 / 16) * nchunk * kWave + wl;

  floatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
  for (int kb0 = 0; kb0 < H; kb0 += kBlockCols) {
    const int cols = min(kBlockCols, H - kb0);
    const int nc = cols / 16;
    // this wave's chunks of the block: [c0, c1), at most kRouteBatch of them
    const int c0 = wave * nc / kRouteWaves, c1 = (wave + 1) * nc / kRouteWaves;
    const int clast = max(c1 - 1, c0);  // in range whenever the wave has chunks
    float4 b[kRouteBatch];
#pragma unroll
    for (int i = 0; i < kRouteBatch; ++i) {
      const int c = kb0 / 16 + min(min(c0 + i, clast), nc - 1);  // chunks past c1 re-read one and go unused
      b[i] = wrow[static_cast<size_t>(c) * kWave];
    }
    // stage rows t0 .. t0+15 (clamped to T-1; those rows are computed and dropped)
    const int pieces_per_row = cols * kEb / 16;
    if (kb0 > 0) __syncthreads();  // the previous block's fragments are consumed
    for (int i = tid; i < 16 * pieces_per_row; i += kRouteThreads) {
      const int row = i / pieces_per_row, q = i % pieces_per_row;
      const int t = min(t0 + row, T - 1);
      const uint4 v = *reinterpret_cast<const uint4*>(reinterpret_cast<const unsigned char*>(hidden) +
                                                      (static_cast<size_t>(t) * H + kb0) * kEb + q * 16);
      *reinterpret_cast<uint4*>(hs + row * kRowBytes + q * 16) = v;
    }
    __syncthreads();
    const unsigned char* arow = hs + r * kRowBytes + 4 * g * kEb;
#pragma unroll
    for (int i = 0; i < kRouteBatch; i += 2) {
      const int ca = min(min(c0 + i, clast), nc - 1), cb = min(min(c0 + i + 1, clast), nc - 1);
      const float4 a0 = widen4(reinterpret_cast<const TIn*>(arow + ca * 16 * kEb));
      const float4 a1 = widen4(reinterpret_cast<const TIn*>(arow + cb * 16 * kEb));
      floatx4 n0 = mfma_f32_16x16x4(a0.x, b[i].x, acc0);
      floatx4 n1 = mfma_f32_16x16x4(a1.x, b[i + 1].x, acc1);
      n0 = mfma_f32_16x16x4(a0.y, b[i].y, n0);
      n1 = mfma_f32_16x16x4(a1.y, b[i + 1].y, n1);
      n0 = mfma_f32_16x16x4(a0.z, b[i].z, n0);
      n1 = mfma_f32_16x16x4(a1.z, b[i + 1].z, n1);
      n0 = mfma_f32_16x16x4(a0.w, b[i].w, n0);
      n1 = mfma_f32_16x16x4(a1.w, b[i + 1].w, n1);
      acc0 = c0 + i < c1 ? n0 : acc0;  // wave-uniform selects, no branch
      acc1 = c0 + i + 1 < c1 ? n1 : acc1;
    }
  }
  floatx4 acc;
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i] = acc0[i] + acc1[i];
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
    const int e = e0 + r;
    if (r < EW && e < E) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int tt = t0 + 4 * g + i;
        if (tt < T) logits[static_cast<size_t>(tt) * E + e] = s[i];
      }
    }
  }
}

}  // namespace

size_t packed_router_bytes(int E, int H) { return static_cast<size_t>((E + 15) / 16) * 16 * H * sizeof(float); }

hipError_t launch_pack_router(const float* src, int E, int H, float* dst, hipStream_t stream) {
  const size_t pieces = packed_router_bytes(E, H) / 16;
  const int block = 256;
  const size_t want = (pieces + block - 1) / block;
  const int grid = static_cast<int>(want < 65536 ? want : 65536);
  pack_router_kernel<<<grid, block, 0, stream>>>(reinterpret_cast<const float4*>(src), reinterpret_cast<float4*>(dst),
                                                 E, H);
  return hipGetLastError();
}

hipError_t launch_route(const void* hidden, int hidden_is_bf16, const float* router_packed, int T, int H, int E,
                        float* logits, hipStream_t stream) {
  const float4* wp = reinterpret_cast<const float4*>(router_packed);
  const int ttiles = (T + 15) / 16;
  // small grids: 8 experts per workgroup, so twice as many CUs read the weights
  const bool half = ((E + 15) / 16) * ttiles < 128;
  if (half) {
    dim3 grid((E + 7) / 8, ttiles);
    if (hidden_is_bf16)
      route_kernel<uint16_t, 8><<<grid, kRouteThreads, 0, stream>>>(static_cast<const uint16_t*>(hidden), wp, T, H,
                                                                     E, logits);
    else
      route_kernel<float, 8><<<grid, kRouteThreads, 0, stream>>>(static_cast<const float*>(hidden), wp, T, H, E,
                                                                  logits);
  } else {
    dim3 grid((E + 15) / 16, ttiles);
    if (hidden_is_bf16)
      route_kernel<uint16_t, 16><<<grid, kRouteThreads, 0, stream>>>(static_cast<const uint16_t*>(hidden), wp, T, H,
                                                                      E, logits);
    else
      route_kernel<float, 16><<<grid, kRouteThreads, 0, stream>>>(static_cast<const float*>(hidden), wp, T, H, E,
                                                                   logits);
  }
  return hipGetLastError();
}

}  // namespace amoe
