// Workgroup residency probe (test infrastructure, not part of the library).
//
// How many workgroups of a given size and static shared-memory footprint
// run on one compute unit at the same time.  Each workgroup fills its
// shared array, runs a fixed chain of FMAs (about 40 us per wave), and its
// first lane records the hardware id of the CU it ran on (HW_ID and XCC_ID
// registers) and the start and end of its run (s_memrealtime).  The host
// counts, per CU, the largest number of overlapping [start, end] intervals.
// The grid holds 8 workgroups per CU; every access stays inside the arrays
// the host allocates for it.
//
// Usage: residency_probe   (prints one line per case)
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <map>
#include <utility>
#include <vector>

struct Rec {
  unsigned hw, xcc;
  unsigned long long t0, t1;
};

template <int BYTES, int NT>
__global__ void __launch_bounds__(NT) probe(Rec* rec, float* sink, int iters) {
  __shared__ float s[BYTES / 4];
  const unsigned long long t0 = __builtin_amdgcn_s_memrealtime();
  for (int i = threadIdx.x; i < BYTES / 4; i += NT) s[i] = (float)i;
  __syncthreads();
  float a = s[(threadIdx.x * 7) % (BYTES / 4)];
  for (int i = 0; i < iters; ++i) a = fmaf(a, 1.0001f, 0.5f);
  __syncthreads();
  const unsigned long long t1 = __builtin_amdgcn_s_memrealtime();
  sink[blockIdx.x * NT + threadIdx.x] = a;
  if (threadIdx.x == 0) {
    Rec r;
    r.hw = __builtin_amdgcn_s_getreg((31 << 11) | 4);    // HW_ID
    r.xcc = __builtin_amdgcn_s_getreg((31 << 11) | 20);  // XCC_ID
    r.t0 = t0;
    r.t1 = t1;
    rec[blockIdx.x] = r;
  }
}

template <int BYTES, int NT>
static bool run(int cus) {
  const int nblk = cus * 8;
  Rec* rec = nullptr;
  float* sink = nullptr;
  if (hipMalloc(&rec, nblk * sizeof(Rec)) != hipSuccess) return false;
  if (hipMalloc(&sink, (size_t)nblk * NT * 4) != hipSuccess) return false;
  hipLaunchKernelGGL((probe<BYTES, NT>), dim3(nblk), dim3(NT), 0, 0, rec, sink, 20000);
  const hipError_t e = hipDeviceSynchronize();
  std::vector<Rec> h(nblk);
  const hipError_t ec = hipMemcpy(h.data(), rec, nblk * sizeof(Rec), hipMemcpyDeviceToHost);
  (void)hipFree(rec);
  (void)hipFree(sink);
  if (e != hipSuccess || ec != hipSuccess) {
    std::printf("threads=%d lds=%d error %s\n", NT, BYTES, hipGetErrorString(e != hipSuccess ? e : ec));
    return false;
  }
  // CU key: XCC, shader engine, shader array, CU
  std::map<unsigned, std::vector<std::pair<unsigned long long, int>>> ev;
  for (const Rec& r : h) {
    const unsigned key = ((r.xcc & 0xF) << 16) | (((r.hw >> 13) & 7) << 8) | (((r.hw >> 12) & 1) << 4) | ((r.hw >> 8) & 0xF);
    ev[key].push_back({r.t0, +1});
    ev[key].push_back({r.t1, -1});
  }
  int most = 0;
  double mean = 0;
  for (auto& kv : ev) {
    auto& v = kv.second;
    std::sort(v.begin(), v.end(), [](const auto& a, const auto& b) {
      return a.first < b.first || (a.first == b.first && a.second < b.second);
    });
    int c = 0, m = 0;
    for (const auto& x : v) m = std::max(m, c += x.second);
    most = std::max(most, m);
    mean += m;
  }
  int api = -1;
  (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(&api, probe<BYTES, NT>, NT, 0);
  std::printf("waves=%d lds=%d cus=%zu resident_max=%d resident_mean=%.2f occupancy_query=%d\n", NT / 64, BYTES,
              ev.size(), most, mean / ev.size(), api);
  std::fflush(stdout);
  return true;
}

template <int NT>
static bool sweep(int cus) {
  return run<28672, NT>(cus) && run<40960, NT>(cus) && run<53248, NT>(cus) && run<57344, NT>(cus) &&
         run<69632, NT>(cus) && run<102400, NT>(cus);
}

int main() {
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0) != hipSuccess || cus <= 0) return 1;
  const bool ok = sweep<64>(cus) && sweep<128>(cus) && sweep<256>(cus) && sweep<320>(cus) && sweep<384>(cus) &&
                  sweep<512>(cus) && sweep<640>(cus);
  return ok ? 0 : 1;
}
