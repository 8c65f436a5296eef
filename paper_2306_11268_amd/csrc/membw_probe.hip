// Practical HBM ceiling for the traffic mixes of the separable layer passes.
//
// Memory-only kernels move a [B][n][n] complex64 field with the access
// pattern and read/write mix of the layer passes, no arithmetic:
//   1R1W  one read, one write per element       (a propagation pass)
//   1R2W  one read, two writes (field + saved)  (forward layer pass)
//   2R1W  two reads (field + saved), one write  (adjoint layer pass)
// over row tiles (16 consecutive rows per workgroup, contiguous) and column
// tiles (T consecutive columns, every 8th row per thread).  Prints one JSON
// object with the time and bytes per second of each case.  Standalone
// program; it shares nothing with the library.
//
//   ./membw_probe [batch=500] [n=200]
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>

namespace {

constexpr int kRowsPerThread = 25;  // 8 row-slots x 25 = 200 rows

template <int T, int NR, int NW>
__global__ void __launch_bounds__(T * 8) col_mix(const float2* __restrict__ a, const float2* __restrict__ b,
                                                 float2* __restrict__ c, float2* __restrict__ d, int n,
                                                 int tiles) {
  const int nt = (n + T - 1) / T;
  const int t = blockIdx.x;
  if (t >= tiles) return;
  const int smp = t / nt;
  const int col = (t - smp * nt) * T + (int)threadIdx.x % T;
  const int s = (int)threadIdx.x / T;
  if (col >= n) return;
  const size_t base = (size_t)smp * n * n;
  float2 x[kRowsPerThread];
#pragma unroll
  for (int k = 0; k < kRowsPerThread; ++k) {
    const int r = s + 8 * k;
    if (r < n) {
      const size_t i = base + (size_t)r * n + col;
      x[k] = a[i];
      if (NR == 2) {
        const float2 y = b[i];
        x[k].x += y.x;
        x[k].y += y.y;
      }
    }
  }
#pragma unroll
  for (int k = 0; k < kRowsPerThread; ++k) {
    const int r = s + 8 * k;
    if (r < n) {
      const size_t i = base + (size_t)r * n + col;
      c[i] = x[k];
      if (NW == 2) d[i] = x[k];
    }
  }
}

template <int NR, int NW>
__global__ void __launch_bounds__(128) row_mix(const float2* __restrict__ a, const float2* __restrict__ b,
                                               float2* __restrict__ c, float2* __restrict__ d, int n, int tiles) {
  const int nt = (n + 15) / 16;
  const int t = blockIdx.x;
  if (t >= tiles) return;
  const int smp = t / nt;
  const int tile = t - smp * nt;
  const int rows = min(16, n - tile * 16);
  const size_t base = (size_t)smp * n * n + (size_t)tile * 16 * n;
  const int total = rows * n;
  float2 x[kRowsPerThread];
#pragma unroll
  for (int k = 0; k < kRowsPerThread; ++k) {
    const int e = (int)threadIdx.x + 128 * k;
    if (e < total) {
      x[k] = a[base + e];
      if (NR == 2) {
        const float2 y = b[base + e];
        x[k].x += y.x;
        x[k].y += y.y;
      }
    }
  }
#pragma unroll
  for (int k = 0; k < kRowsPerThread; ++k) {
    const int e = (int)threadIdx.x + 128 * k;
    if (e < total) {
      c[base + e] = x[k];
      if (NW == 2) d[base + e] = x[k];
    }
  }
}

template <class F>
double time_us(F f) {
  hipEvent_t e0, e1;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) std::exit(1);
  for (int i = 0; i < 3; ++i) f();
  (void)hipEventRecord(e0, nullptr);
  constexpr int reps = 10;
  for (int i = 0; i < reps; ++i) f();
  (void)hipEventRecord(e1, nullptr);
  (void)hipEventSynchronize(e1);
  float ms = 0.f;
  (void)hipEventElapsedTime(&ms, e0, e1);
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  return 1e3 * ms / reps;
}

}  // namespace

int main(int argc, char** argv) {
  const int batch = argc > 1 ? std::atoi(argv[1]) : 500;
  const int n = argc > 2 ? std::atoi(argv[2]) : 200;
  if (batch < 1 || n < 1 || n > 8 * kRowsPerThread) {
    std::fprintf(stderr, "batch >= 1 and 1 <= n <= %d\n", 8 * kRowsPerThread);
    return 2;
  }
  const size_t el = (size_t)batch * n * n;
  float2 *a = nullptr, *b = nullptr, *c = nullptr, *d = nullptr;
  if (hipMalloc(&a, el * 8) != hipSuccess || hipMalloc(&b, el * 8) != hipSuccess ||
      hipMalloc(&c, el * 8) != hipSuccess || hipMalloc(&d, el * 8) != hipSuccess) {
    std::fprintf(stderr, "allocation failed\n");
    return 1;
  }
  (void)hipMemset(a, 0, el * 8);
  (void)hipMemset(b, 0, el * 8);
  const int rt = batch * ((n + 15) / 16);
  const int c16 = batch * ((n + 15) / 16);
  const int c32 = batch * ((n + 31) / 32);
  struct Case {
    const char* name;
    int elements_moved;  // reads + writes per field element
    double us;
  } cases[] = {
      {"row_1R1W", 2, time_us([&] { row_mix<1, 1><<<rt, 128>>>(a, b, c, d, n, rt); })},
      {"col16_1R1W", 2, time_us([&] { col_mix<16, 1, 1><<<c16, 128>>>(a, b, c, d, n, c16); })},
      {"row_1R2W", 3, time_us([&] { row_mix<1, 2><<<rt, 128>>>(a, b, c, d, n, rt); })},
      {"col16_1R2W", 3, time_us([&] { col_mix<16, 1, 2><<<c16, 128>>>(a, b, c, d, n, c16); })},
      {"col32_1R2W", 3, time_us([&] { col_mix<32, 1, 2><<<c32, 256>>>(a, b, c, d, n, c32); })},
      {"row_2R1W", 3, time_us([&] { row_mix<2, 1><<<rt, 128>>>(a, b, c, d, n, rt); })},
      {"col16_2R1W", 3, time_us([&] { col_mix<16, 2, 1><<<c16, 128>>>(a, b, c, d, n, c16); })},
      {"col32_2R1W", 3, time_us([&] { col_mix<32, 2, 1><<<c32, 256>>>(a, b, c, d, n, c32); })},
  };
  if (hipDeviceSynchronize() != hipSuccess) return 1;
  std::printf("{\"batch\": %d, \"n\": %d, \"field_bytes\": %zu", batch, n, el * 8);
  for (const Case& k : cases) {
    const double bytes = (double)k.elements_moved * el * 8;
    std::printf(", \"%s\": {\"us\": %.1f, \"GBps\": %.0f}", k.name, k.us, bytes / k.us / 1e3);
  }
  std::printf("}\n");
  (void)hipFree(a);
  (void)hipFree(b);
  (void)hipFree(c);
  (void)hipFree(d);
  return 0;
}
