// Read-bandwidth probe for gfx950: how fast HBM delivers a (N, H, D) point array when each
// workgroup reads only one head's segment of every row (the access of the streaming passes,
// which own one (sample, head) per workgroup), against workgroups that read whole rows. One
// 512 MiB buffer; rows of 1024 B (fp32, H = 8, D = 32) and 512 B (bf16); segments of 128 B
// and 64 B. The same number of workgroups (4096, 256 threads) and the same bytes in every
// case; each thread keeps eight 16-byte loads in flight. A second numbering gives the
// segment readers of one row block workgroup numbers that are equal mod 8, so they share one
// XCD and its L2. Not part of the library.
//
//   hipcc --offload-arch=gfx950 -O3 -Xclang -target-feature -Xclang -packed-fp32-ops \
//       -o rowseg paper_2609_32525_amd/probes/rowseg.hip && ./rowseg
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>

typedef float f4 __attribute__((ext_vector_type(4)));

// Workgroup -> (chunk, segment): plain, segment = blockIdx % nseg and chunk = blockIdx / nseg
// (consecutive workgroups, which the dispatcher deals round-robin to the 8 XCDs, read the
// segments of one chunk); XCD-grouped, the nseg segments of one chunk go to workgroups
// b, b + 8, b + 16, ..., all on the same XCD. The chunk's rows are
// [chunk * rpw, min(nrows, (chunk + 1) * rpw)). Thread t reads 16-byte column t % seg_f4 of
// the segment in rows t / seg_f4, + 256 / seg_f4, ...
__global__ __launch_bounds__(256) void k_rows(const f4* __restrict__ p, int64_t nrows, int row_f4,
                                              int seg_f4, int nseg, int64_t rpw, int xcd,
                                              float* out) {
  const int b = blockIdx.x, x = b % 8, k = b / 8;
  const int seg = xcd ? k % nseg : b % nseg;
  const int64_t chunk = xcd ? (int64_t)(k / nseg) * 8 + x : b / nseg;
  const int64_t r0 = chunk * rpw, r1 = r0 + rpw < nrows ? r0 + rpw : nrows;
  const int t = threadIdx.x, step = 256 / seg_f4;
  const f4* q = p + seg * seg_f4 + t % seg_f4;
  f4 acc{0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
  for (int64_t r = r0 + t / seg_f4; r < r1; r += step) acc += q[r * row_f4];
  out[blockIdx.x * 256 + t] = acc[0] + acc[1] + acc[2] + acc[3];
}

#define CK(x)                                                                  \
  do {                                                                         \
    hipError_t e_ = (x);                                                       \
    if (e_ != hipSuccess) {                                                    \
      std::printf("%s failed: %s\n", #x, hipGetErrorString(e_));               \
      return 1;                                                                \
    }                                                                          \
  } while (0)

int main() {
  const size_t bytes = (size_t)512 << 20;
  const int blocks = 4096;
  f4* buf = nullptr;
  float* out = nullptr;
  CK(hipMalloc(&buf, bytes));
  CK(hipMalloc(&out, (size_t)blocks * 256 * sizeof(float)));
  CK(hipMemset(buf, 0, bytes));
  hipEvent_t e0, e1;
  CK(hipEventCreate(&e0));
  CK(hipEventCreate(&e1));
  struct Case {
    const char* name;
    int row_bytes, seg_bytes, xcd;
  } cases[] = {{"fp32 rows 1024 B, whole rows", 1024, 1024, 0},
               {"fp32 rows 1024 B, one 128 B head segment per workgroup", 1024, 128, 0},
               {"fp32 rows 1024 B, 128 B segments, XCD-grouped", 1024, 128, 1},
               {"bf16 rows 512 B, whole rows", 512, 512, 0},
               {"bf16 rows 512 B, one 64 B head segment per workgroup", 512, 64, 0},
               {"bf16 rows 512 B, 64 B segments, XCD-grouped", 512, 64, 1}};
  for (const Case& c : cases) {
    const int row_f4 = c.row_bytes / 16, seg_f4 = c.seg_bytes / 16, nseg = c.row_bytes / c.seg_bytes;
    const int64_t nrows = (int64_t)(bytes / c.row_bytes);
    const int64_t chunks = blocks / nseg;
    const int64_t rpw = (nrows + chunks - 1) / chunks;
    // every index stays below nrows * row_f4: r < nrows and seg * seg_f4 + seg_f4 <= row_f4
    if (256 % seg_f4 != 0 || chunks * nseg != blocks || rpw * chunks < nrows) return 2;
    if (c.xcd && blocks % (8 * nseg) != 0) return 2;  // then chunk = (k / nseg) * 8 + x < chunks
    for (int w = 0; w < 3; ++w)
      hipLaunchKernelGGL(k_rows, dim3(blocks), dim3(256), 0, 0, buf, nrows, row_f4, seg_f4, nseg,
                         rpw, c.xcd, out);
    CK(hipGetLastError());
    const int iters = 20;
    CK(hipEventRecord(e0, 0));
    for (int it = 0; it < iters; ++it)
      hipLaunchKernelGGL(k_rows, dim3(blocks), dim3(256), 0, 0, buf, nrows, row_f4, seg_f4, nseg,
                         rpw, c.xcd, out);
    CK(hipEventRecord(e1, 0));
    CK(hipEventSynchronize(e1));
    float ms = 0.f;
    CK(hipEventElapsedTime(&ms, e0, e1));
    std::printf("%-56s %8.1f GB/s  (%.1f us per 512 MiB read)\n", c.name,
                (double)bytes * iters / (ms * 1e-3) / 1e9, ms * 1e3 / iters);
  }
  CK(hipFree(buf));
  CK(hipFree(out));
  return 0;
}
