// Small stream kernels around the layer: the row copy that joins the outputs of
// a block served in waves (expert offload) and the residual add that chains
// stacked verify layers.
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

}  // namespace

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
