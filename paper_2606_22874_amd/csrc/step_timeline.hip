// Timeline build of the fused decode step -- a measurement tool, not part of
// libspot.so.  The step kernel's phase hooks stamp the 100 MHz real-time
// counter (s_memrealtime, one clock for the whole device) into device
// arrays, one row per workgroup, with the XCD the workgroup ran on:
//   step phases  0 start, 1 own scoring done, 2 selection core done (a
//                row's selecting workgroup; the bitmap goes out right after),
//                3 selection written, 4 attention start (set received),
//                5 attention done, 6 completion counter bumped, 7 merged
//                (the pair's last workgroup);
//   selection    0 core entered, 1 this wave's scores in, 2 every wave's
//                scores in (after the first barrier), 6 histogram, 7 bin
//                scan, 8 members packed, 3 survivors, 5 survivors packed
//                and 9 ranked (the nucleus cut of at most 64 survivors),
//                4 core done.
// Everything else is step.hip compiled unchanged; paper_2606_22874_amd/
// step_timeline.py links this object with the library's other objects.
#include <hip/hip_runtime.h>

constexpr int kTimelineWgs = 4096;
__device__ unsigned long long g_step_ts[kTimelineWgs][8];
__device__ unsigned long long g_sel_ts[kTimelineWgs][10];
__device__ unsigned g_step_xcc[kTimelineWgs];

#define SPOT_STEP_TS(i)                                                        \
  do {                                                                         \
    if (threadIdx.x == 0 && blockIdx.x < kTimelineWgs) {                       \
      g_step_ts[blockIdx.x][i] = __builtin_amdgcn_s_memrealtime();             \
      if ((i) == 0) {                                                          \
        unsigned x;                                                            \
        asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));       \
        g_step_xcc[blockIdx.x] = x;                                            \
      }                                                                        \
    }                                                                          \
  } while (0)
#define SPOT_SEL_TS(i)                                                         \
  do {                                                                         \
    if (threadIdx.x == 0 && blockIdx.x < kTimelineWgs)                         \
      g_sel_ts[blockIdx.x][i] = __builtin_amdgcn_s_memrealtime();              \
  } while (0)

// The workloads this tool stamps have 4 query heads per KV head.
#define SPOT_STEP_GROUP4_ONLY
#include "step.hip"

extern "C" {

// Copies the stamps to host arrays of kTimelineWgs x 8 / x 10 uint64 and
// kTimelineWgs uint32; returns a hipError_t.
int spot_timeline_read(unsigned long long* step_ts, unsigned long long* sel_ts, unsigned* xcc) {
  hipError_t e = hipMemcpyFromSymbol(step_ts, HIP_SYMBOL(g_step_ts), sizeof(g_step_ts));
  if (e == hipSuccess) e = hipMemcpyFromSymbol(sel_ts, HIP_SYMBOL(g_sel_ts), sizeof(g_sel_ts));
  if (e == hipSuccess) e = hipMemcpyFromSymbol(xcc, HIP_SYMBOL(g_step_xcc), sizeof(g_step_xcc));
  return (int)e;
}

// Zeroes the stamps (0 = phase not reached).
int spot_timeline_clear() {
  static unsigned long long zero[kTimelineWgs][10];
  hipError_t e = hipMemcpyToSymbol(HIP_SYMBOL(g_step_ts), zero, sizeof(g_step_ts));
  if (e == hipSuccess) e = hipMemcpyToSymbol(HIP_SYMBOL(g_sel_ts), zero, sizeof(g_sel_ts));
  return (int)e;
}

int spot_timeline_capacity() { return kTimelineWgs; }

}  // extern "C"
