// Vector-ALU rate probe for gfx950: throughput of v_exp_f32 and of v_add_f32 with eight
// independent chains per lane and 4096 workgroups of 256 threads (16 per compute unit), so
// that issue rate, not latency, bounds both. It gives the measured side of the VALU figures
// the profiling summaries use (128 fp32 lanes per clock per compute unit, transcendentals at a
// quarter of that). Not part of the library.
//
//   hipcc --offload-arch=gfx950 -O3 -Xclang -target-feature -Xclang -packed-fp32-ops \
//       -o vrate paper_2609_32525_amd/probes/vrate.hip && ./vrate
#include <hip/hip_runtime.h>

#include <cstdio>

template <int OP>
__global__ __launch_bounds__(256) void k_rate(float* out, int iters, float seed) {
  float x[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) x[c] = seed + c * 1e-3f + threadIdx.x * 1e-6f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < 8; ++c) x[c] = OP == 0 ? __builtin_amdgcn_exp2f(x[c]) : x[c] + 1.0f;
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < 8; ++c) s += x[c];
  out[blockIdx.x * 256 + threadIdx.x] = s;  // one value per thread: grid * 256 floats
}

int main() {
  const int blocks = 4096, iters = 4096;
  float* out = nullptr;
  if (hipMalloc(&out, sizeof(float) * blocks * 256) != hipSuccess) return 1;
  hipEvent_t a, b;
  if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess) return 1;
  for (int op = 0; op < 2; ++op) {
    for (int rep = 0; rep < 3; ++rep) {
      if (hipEventRecord(a) != hipSuccess) return 1;
      if (op == 0)
        hipLaunchKernelGGL(k_rate<0>, dim3(blocks), dim3(256), 0, 0, out, iters, -100.f);
      else
        hipLaunchKernelGGL(k_rate<1>, dim3(blocks), dim3(256), 0, 0, out, iters, 0.f);
      if (hipEventRecord(b) != hipSuccess || hipEventSynchronize(b) != hipSuccess) return 1;
      float ms = 0.f;
      if (hipEventElapsedTime(&ms, a, b) != hipSuccess) return 1;
      const double n = (double)blocks * 256 * 8 * iters;
      std::printf("%s rep %d: %.3f ms, %.2f T lane-ops/s\n", op == 0 ? "v_exp_f32" : "v_add_f32",
                  rep, ms, n / (ms * 1e-3) / 1e12);
    }
  }
  if (hipGetLastError() != hipSuccess) return 2;
  return hipFree(out) == hipSuccess ? 0 : 1;
}
