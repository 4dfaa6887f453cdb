// Small stream kernels around the layer: the row copy that joins the outputs of
// a block served in waves (expert offload), the residual add that chains
// stacked verify layers, and a plain streaming read that measures the HBM
// read rate the expert-weight stream is compared with.
#include "common.hpp"
#include "launch.hpp"

namespace amoe {

namespace {

// out = hidden + y, rounded to the hidden dtype (bf16: fp32 sum, then round to
// nearest even), four elements per thread
template <bool kBf16>
__global__ void residual_add_kernel(const void* __restrict__ hidden, const float4* __restrict__ y,
                                    void* __restrict__ out, size_t n4) {
  for (size_t i = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; i < n4;
       i += static_cast<size_t>(gridDim.x) * blockDim.x) {
    const float4 v = y[i];
    if (kBf16) {
      const uint2 h = static_cast<const uint2*>(hidden)[i];
      const float a0 = __uint_as_float(h.x << 16) + v.x, a1 = __uint_as_float(h.x & 0xffff0000u) + v.y;
      const float a2 = __uint_as_float(h.y << 16) + v.z, a3 = __uint_as_float(h.y & 0xffff0000u) + v.w;
      static_cast<uint2*>(out)[i] =
          make_uint2(float_to_bf16_bits(a0) | (static_cast<uint32_t>(float_to_bf16_bits(a1)) << 16),
                     float_to_bf16_bits(a2) | (static_cast<uint32_t>(float_to_bf16_bits(a3)) << 16));
    } else {
      const float4 h = static_cast<const float4*>(hidden)[i];
      static_cast<float4*>(out)[i] = make_float4(h.x + v.x, h.y + v.y, h.z + v.z, h.w + v.w);
    }
  }
}

// dst[t, :] = src[t, :] for the rows whose tag equals `tag` (float4 columns)
__global__ void copy_rows_kernel(const float4* __restrict__ src, float4* __restrict__ dst,
                                 const int32_t* __restrict__ row_tag, int tag, int T, int H4) {
  const int t = blockIdx.y;
  if (t >= T || row_tag[t] != tag) return;
  for (int c = blockIdx.x * blockDim.x + threadIdx.x; c < H4; c += gridDim.x * blockDim.x)
    dst[static_cast<size_t>(t) * H4 + c] = src[static_cast<size_t>(t) * H4 + c];
}

// XOR of the 16-byte pieces [b per, (b + 1) per) of src (clamped to n16) into
// sink[b], for workgroup b: eight non-temporal loads in flight per thread
// before any is used, the access pattern of a weight stream without the
// arithmetic.  The XOR keeps every load live.
__global__ __launch_bounds__(256) void stream_read_kernel(const uint4* __restrict__ src, size_t n16, size_t per,
                                                         uint32_t* __restrict__ sink) {
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  constexpr int kU = 8;
  const size_t base = blockIdx.x * per;
  const size_t end = base + per < n16 ? base + per : n16;
  uint32_t acc = 0u;
  for (size_t i = base + threadIdx.x; i < end; i += 256 * kU) {
    u32x4 v[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const size_t j = i + static_cast<size_t>(u) * 256;
      v[u] = j < end ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src + j)) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  __shared__ uint32_t part[4];
  for (int o = 32; o >= 1; o >>= 1) acc ^= __shfl_xor(acc, o);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = part[0] ^ part[1] ^ part[2] ^ part[3];
}

}  // namespace

hipError_t launch_stream_read(const void* src, size_t bytes, uint32_t* sink, int grid, hipStream_t stream) {
  const size_t n16 = bytes / 16;
  const size_t per = (n16 + grid - 1) / grid;
  stream_read_kernel<<<grid, 256, 0, stream>>>(static_cast<const uint4*>(src), n16, per, sink);
  return hipGetLastError();
}

hipError_t launch_copy_rows(const float* src, float* dst, const int32_t* row_tag, int tag, int T, int H,
                            hipStream_t stream) {
  if (H % 4 != 0) return hipErrorInvalidValue;
  const int H4 = H / 4;
  copy_rows_kernel<<<dim3((H4 + 255) / 256, T), 256, 0, stream>>>(reinterpret_cast<const float4*>(src),
                                                                 reinterpret_cast<float4*>(dst), row_tag, tag, T, H4);
  return hipGetLastError();
}

hipError_t launch_residual_add(const void* hidden, int is_bf16, const float* y, int T, int H, void* out,
                               hipStream_t stream) {
  const size_t n4 = static_cast<size_t>(T) * H / 4;
  const int block = 256;
  const size_t want = (n4 + block - 1) / block;
  const int grid = static_cast<int>(want < 4096 ? want : 4096);
  if (is_bf16)
    residual_add_kernel<true><<<grid, block, 0, stream>>>(hidden, reinterpret_cast<const float4*>(y), out, n4);
  else
    residual_add_kernel<false><<<grid, block, 0, stream>>>(hidden, reinterpret_cast<const float4*>(y), out, n4);
  return hipGetLastError();
}

}  // namespace amoe
