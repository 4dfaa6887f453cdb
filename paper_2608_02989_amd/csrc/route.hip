// Router logits z_t = W_r h_t (Sec. 3.1): a [T,H] x [E,H]^T product in fp32
// accuracy, one 16-token x 16-expert tile (or 16 x 8 for small grids) per
// workgroup of 16 waves, each wave reducing a slice of H.
//
// The fp32 router matrix is stored as three bf16 planes, hi = bf16(w),
// mid = bf16(w - hi), lo = bf16(w - hi - mid), whose sum is w exactly for
// every |w| between about 1e-33 and 3.39e38 (below, the remainders leave the
// normal range and the loss is under 2^-125 per weight; above, the largest
// bf16 is exceeded and hi is infinite).  A bf16 hidden state then takes
// the bf16 MFMA (v_mfma_f32_16x16x32_bf16) three times per chunk, once per
// plane, with exact products and fp32 accumulation: three instructions that
// together run about five times faster than the fp32 MFMA they replace,
// which is the bound of this small product on the few CUs it occupies.  An
// fp32 hidden state rebuilds w in registers (exact) and uses the fp32 MFMA.
//
// Both operands are read with whole-cache-line accesses: each plane comes in
// MFMA fragment order (one contiguous 1 KiB read per 16-expert x 32-column
// chunk, see acceptmoe_pack_router_weights), and the workgroup's 16 hidden
// rows are staged in LDS with row-contiguous loads.  Every thread issues its
// weight loads and all of its staging loads before it waits for any of them,
// so one memory round trip covers a staged block.  The 16 partial tiles are
// summed in LDS in a fixed order (deterministic).
#include "common.hpp"
#include "launch.hpp"

namespace amoe {

namespace {

constexpr int kRouteWaves = 16;
constexpr int kRouteThreads = kRouteWaves * kWave;
constexpr int kRouteStageBytes = 64 * 1024;  // hidden bytes staged per block (16 rows)
constexpr int kRouteStageLoads = kRouteStageBytes / 16 / kRouteThreads;  // 16-byte loads per thread and block
constexpr int kRouteRowPad = 16;             // bytes appended to each staged row (LDS banks)
constexpr int kRoutePlanes = 3;              // hi, mid, lo
constexpr int kRouteChunk = 32;              // columns per packed chunk

__device__ __forceinline__ float bits_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bits_hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }

// Packed router: rows padded with zeros to a multiple of 16, columns to a
// multiple of 32.  Fragment (expert tile et, chunk c, plane p) holds, for
// lane L = n + 16 g, plane p of the eight weights of row 16 et + n, columns
// 32 c + 8 g .. +7, as bf16 (16 bytes).  One thread writes one lane of the
// three planes of a chunk.
__global__ void pack_router_kernel(const float* __restrict__ src, uint4* __restrict__ dst, int E, int H) {
  const int nchunk = (H + kRouteChunk - 1) / kRouteChunk;
  const size_t total = static_cast<size_t>((E + 15) / 16) * nchunk * kWave;
  for (size_t q = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; q < total;
       q += static_cast<size_t>(gridDim.x) * blockDim.x) {
    const int lane = static_cast<int>(q & 63);
    const size_t f = q >> 6;
    const int c = static_cast<int>(f % nchunk);
    const int et = static_cast<int>(f / nchunk);
    const int row = et * 16 + (lane & 15);
    const int col = c * kRouteChunk + 8 * (lane >> 4);
    float w[8];
    if (row < E && col < H) {  // H % 16 == 0: the eight columns are all inside or all outside
      const float4* s4 = reinterpret_cast<const float4*>(src + static_cast<size_t>(row) * H + col);
      const float4 u = s4[0], v = s4[1];
      w[0] = u.x; w[1] = u.y; w[2] = u.z; w[3] = u.w;
      w[4] = v.x; w[5] = v.y; w[6] = v.z; w[7] = v.w;
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) w[j] = 0.f;
    }
    uint32_t pl[kRoutePlanes][4];
#pragma unroll
    for (int j = 0; j < 8; j += 2) {
      uint32_t hw[2][kRoutePlanes];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        float rest = w[j + u];
#pragma unroll
        for (int p = 0; p < kRoutePlanes; ++p) {
          const uint16_t b = float_to_bf16_bits(rest);
          hw[u][p] = b;
          rest = rest - __uint_as_float(static_cast<uint32_t>(b) << 16);
        }
      }
#pragma unroll
      for (int p = 0; p < kRoutePlanes; ++p) pl[p][j / 2] = hw[0][p] | (hw[1][p] << 16);
    }
#pragma unroll
    for (int p = 0; p < kRoutePlanes; ++p)
      dst[(f * kRoutePlanes + p) * kWave + lane] = make_uint4(pl[p][0], pl[p][1], pl[p][2], pl[p][3]);
  }
}

// grid (ceil(E/EW), ceil(T/16)), block 1024, EW = 16 or 8 experts per
// workgroup.  Lane (r, g) of a wave: token row t0 + r of the A tile and expert
// row r of the B tile; K slice g of chunk c is columns 32c + 8g .. +7 for both
// operands.  With EW = 8 a workgroup reads one half of each 16-row fragment
// (rows 0-7 or 8-15: four whole 128-byte lines of the 1 KiB fragment), lanes
// r >= 8 repeat lanes r - 8 and their output columns are dropped; twice the
// workgroups then share the weights, which matters when only a few tiles
// exist (the per-CU read rate bounds a small grid).
template <typename TIn, int EW>
__global__ __launch_bounds__(kRouteThreads) void route_kernel(const TIn* __restrict__ hidden,
                                                             const uint4* __restrict__ wp, int T, int H, int E,
                                                             float* __restrict__ logits) {
  constexpr int kEb = sizeof(TIn);
  constexpr int kBlockCols = kRouteStageBytes / (16 * kEb);          // staged columns per block
  constexpr int kBatch = kBlockCols / kRouteChunk / kRouteWaves;     // chunks per wave and block
  constexpr int kRowBytes = kBlockCols * kEb + kRouteRowPad;
  static_assert(kBatch >= 1 && kRouteStageLoads * kRouteThreads * 16 == kRouteStageBytes, "staging shape");
  __shared__ __align__(16) unsigned char hs[16 * kRowBytes];
  __shared__ floatx4 part[kRouteWaves][kWave];
  const int tid = threadIdx.x;
  const int wave = wave_id();
  const int lane = lane_id();
  const int r = lane & 15, g = lane >> 4;
  const int e0 = blockIdx.x * EW, t0 = blockIdx.y * 16;
  const int nchunk = (H + kRouteChunk - 1) / kRouteChunk;
  const int Hp = nchunk * kRouteChunk;
  // fragment lane holding expert row (e0 % 16) + (r % EW) for K slice g
  const int wl = (e0 % 16) + (r % EW) + 16 * g;
  const uint4* wrow = wp + static_cast<size_t>(e0 / 16) * nchunk * kRoutePlanes * kWave + wl;

  floatx4 acc[kRoutePlanes];
#pragma unroll
  for (int p = 0; p < kRoutePlanes; ++p) acc[p] = floatx4{0.f, 0.f, 0.f, 0.f};
  for (int kb0 = 0; kb0 < Hp; kb0 += kBlockCols) {
    const int cols = min(kBlockCols, Hp - kb0);  // a multiple of 32
    const int nc = cols / kRouteChunk;
    // this wave's chunks of the block: [c0, c1), at most kBatch of them
    const int c0 = wave * nc / kRouteWaves, c1 = (wave + 1) * nc / kRouteWaves;
    const int clast = max(c1 - 1, c0);  // in range whenever the wave has chunks
    uint4 b[kBatch][kRoutePlanes];
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
      const int c = kb0 / kRouteChunk + min(min(c0 + i, clast), nc - 1);  // chunks past c1 re-read one, unused
#pragma unroll
      for (int p = 0; p < kRoutePlanes; ++p) b[i][p] = wrow[(static_cast<size_t>(c) * kRoutePlanes + p) * kWave];
    }
    // stage rows t0 .. t0+15 (clamped to T-1; those rows are computed and
    // dropped); columns past H (padding to a multiple of 32) are zeros
    const int pieces_per_row = cols * kEb / 16;
    const int npieces = 16 * pieces_per_row;
    uint4 v[kRouteStageLoads];
#pragma unroll
    for (int s = 0; s < kRouteStageLoads; ++s) {
      const int i = tid + s * kRouteThreads;
      const int row = i / pieces_per_row, q = i % pieces_per_row;
      const int col = kb0 + q * (16 / kEb);
      v[s] = make_uint4(0u, 0u, 0u, 0u);
      if (i < npieces && col < H) {
        const int t = min(t0 + row, T - 1);
        v[s] = *reinterpret_cast<const uint4*>(reinterpret_cast<const unsigned char*>(hidden) +
                                               (static_cast<size_t>(t) * H + col) * kEb);
      }
    }
    if (kb0 > 0) __syncthreads();  // the previous block's fragments are consumed
#pragma unroll
    for (int s = 0; s < kRouteStageLoads; ++s) {
      const int i = tid + s * kRouteThreads;
      if (i < npieces)
        *reinterpret_cast<uint4*>(hs + (i / pieces_per_row) * kRowBytes + (i % pieces_per_row) * 16) = v[s];
    }
    __syncthreads();
    const unsigned char* arow = hs + r * kRowBytes + 8 * g * kEb;
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
      const int ci = min(min(c0 + i, clast), nc - 1);
      const unsigned char* ap = arow + ci * kRouteChunk * kEb;
      floatx4 n[kRoutePlanes];
      if constexpr (kEb == 2) {
        const uint4 a = *reinterpret_cast<const uint4*>(ap);
#pragma unroll
        for (int p = 0; p < kRoutePlanes; ++p) n[p] = mfma_bf16_16x16x32(a, b[i][p], acc[p]);
      } else {
        const float4 a0 = *reinterpret_cast<const float4*>(ap);
        const float4 a1 = *reinterpret_cast<const float4*>(ap + 16);
        const float a[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
        const uint32_t* h32 = reinterpret_cast<const uint32_t*>(&b[i][0]);
        const uint32_t* m32 = reinterpret_cast<const uint32_t*>(&b[i][1]);
        const uint32_t* l32 = reinterpret_cast<const uint32_t*>(&b[i][2]);
        n[0] = acc[0];
        n[1] = acc[1];
        n[2] = acc[2];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int q = j >> 1;
          const float w = (j & 1) ? (bits_hi(h32[q]) + bits_hi(m32[q])) + bits_hi(l32[q])
                                  : (bits_lo(h32[q]) + bits_lo(m32[q])) + bits_lo(l32[q]);
          n[j & 1] = mfma_f32_16x16x4(a[j], w, n[j & 1]);
        }
      }
#pragma unroll
      for (int p = 0; p < kRoutePlanes; ++p) acc[p] = c0 + i < c1 ? n[p] : acc[p];  // wave-uniform select
    }
  }
  floatx4 accs;
#pragma unroll
  for (int i = 0; i < 4; ++i) accs[i] = (acc[2][i] + acc[1][i]) + acc[0][i];
  part[wave][lane] = accs;
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

size_t packed_router_bytes(int E, int H) {
  return static_cast<size_t>((E + 15) / 16) * 16 * ((H + kRouteChunk - 1) / kRouteChunk) * kRouteChunk *
         kRoutePlanes * sizeof(uint16_t);
}

hipError_t launch_pack_router(const float* src, int E, int H, void* dst, hipStream_t stream) {
  const size_t pieces = packed_router_bytes(E, H) / (16 * kRoutePlanes);  // one thread per lane of a chunk
  const int block = 256;
  const size_t want = (pieces + block - 1) / block;
  const int grid = static_cast<int>(want < 65536 ? want : 65536);
  pack_router_kernel<<<grid, block, 0, stream>>>(src, static_cast<uint4*>(dst), E, H);
  return hipGetLastError();
}

hipError_t launch_route(const void* hidden, int hidden_is_bf16, const void* router_packed, int T, int H, int E,
                        float* logits, hipStream_t stream) {
  const uint4* wp = static_cast<const uint4*>(router_packed);
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
