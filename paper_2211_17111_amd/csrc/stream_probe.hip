// Measurement probe (not part of the bevpool ABI): a streaming kernel with
// a given mix of bytes read and written, the bandwidth one launch of that
// size and mix reaches on this device.  bench.py times it beside the
// forward, whose algorithmic traffic it matches.
//
// out (n_out 16-byte vectors) receives, for each j, the sum of in[j],
// in[j + n_out], in[j + 2 n_out], ... (every in vector read once, every out
// vector written once; consecutive lanes touch consecutive vectors).

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace {

typedef float float4_t __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void k_stream_mix(const float4_t* __restrict__ in, int64_t n_in,
                                                    float4_t* __restrict__ out, int64_t n_out) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n_out; j += stride) {
    float4_t acc = {0.f, 0.f, 0.f, 0.f};
    for (int64_t i = j; i < n_in; i += n_out) acc += in[i];
    out[j] = acc;
  }
}

}  // namespace

extern "C" int bevpool_probe_stream(const void* in, size_t in_bytes, void* out, size_t out_bytes,
                                    void* stream) {
  const int64_t n_in = (int64_t)(in_bytes / 16), n_out = (int64_t)(out_bytes / 16);
  if (in == nullptr || out == nullptr || n_in < 1 || n_out < 1 ||
      (reinterpret_cast<uintptr_t>(in) & 15u) || (reinterpret_cast<uintptr_t>(out) & 15u))
    return -1;
  const int64_t blocks = (n_out + 255) / 256;
  k_stream_mix<<<dim3((unsigned)(blocks < 65536 ? blocks : 65536)), dim3(256), 0,
                 static_cast<hipStream_t>(stream)>>>(static_cast<const float4_t*>(in), n_in,
                                                     static_cast<float4_t*>(out), n_out);
  return hipGetLastError() == hipSuccess ? 0 : -5;
}
