// Sustained bf16 matrix-core rate of the device, as a measurement reference
// for the attention kernels (not part of the method; built into its own
// library, libconduit_ceiling.so, which only the benchmark loads).
//
// Every wave keeps four independent v_mfma_f32_32x32x16_bf16 accumulations
// going over eight A and eight B operands per lane read once from `ops`
// (random data: the shader clock under matrix-core load depends on the
// operand bits, so the operands should look like real activations).  Two
// waves per SIMD, one 256-thread workgroup per two SIMDs.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kOps = 8;  // A and B operands per lane

__global__ __launch_bounds__(256) void mfma_ceiling_kernel(const u32x4 *ops, float *out, int iters) {
  const int64_t lane_id = (int64_t)blockIdx.x * 256 + threadIdx.x;
  bf16x8 a[kOps], b[kOps];
#pragma unroll
  for (int i = 0; i < kOps; ++i) {
    a[i] = __builtin_bit_cast(bf16x8, ops[lane_id * 2 * kOps + i]);
    b[i] = __builtin_bit_cast(bf16x8, ops[lane_id * 2 * kOps + kOps + i]);
  }
  f32x16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < kOps; i += 2) {
      c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[i], c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i + 1], b[i], c1, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[i + 1], c2, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i + 1], b[i + 1], c3, 0, 0, 0);
    }
  }
  float acc = 0.f;
#pragma unroll
  for (int j = 0; j < 16; ++j) acc += c0[j] + c1[j] + c2[j] + c3[j];
  out[lane_id] = acc;  // keeps the products live
}

}  // namespace

extern "C" {

// Bytes of random operands `conduit_ceiling_mfma_bf16` reads for `blocks`
// workgroups (16-byte bf16x8 values, 2 * 8 per lane).
int64_t conduit_ceiling_ops_bytes(int32_t blocks) { return (int64_t)blocks * 256 * 2 * kOps * 16; }

// FLOP one launch performs.
double conduit_ceiling_flop(int32_t blocks, int32_t iters) {
  return (double)blocks * (256 / 64) * iters * kOps * 2 * 2.0 * 32 * 32 * 16;
}

// Enqueues the measurement kernel on `stream`: `ops` (device, 16-byte
// aligned, conduit_ceiling_ops_bytes(blocks) bytes of bf16), `out` (device,
// blocks * 256 floats).  Returns a hipError_t value (0 on success).
int conduit_ceiling_mfma_bf16(const void *ops, float *out, int32_t blocks, int32_t iters, hipStream_t stream) {
  if (!ops || !out || blocks < 1 || iters < 1 || (reinterpret_cast<uintptr_t>(ops) & 15)) return (int)hipErrorInvalidValue;
  mfma_ceiling_kernel<<<blocks, 256, 0, stream>>>(static_cast<const u32x4 *>(ops), out, iters);
  return (int)hipGetLastError();
}

}  // extern "C"
