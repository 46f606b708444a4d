// Calibration, not part of libmalt: the sustained bf16 matrix-core rate of
// this GPU when nothing but MFMAs run, and the shader clock it runs at, for a
// given instruction (v_mfma_f32_32x32x16_bf16 or v_mfma_f32_16x16x32_bf16) and
// kind of operands.
//
// MI355X's dense bf16 figure (2.5 PFLOP/s) assumes the 2.4 GHz clock. Under
// load the chip is held to its power budget, and the matrix cores' power
// depends on the operand bits and on the instruction: with random operands
// the clock, and with it the attainable rate, falls below the figure. This
// measures that ceiling: 8 waves per CU (2 per SIMD), each cycling
// independent accumulators (8 of 32 x 32, or 16 of 16 x 16) through 8 x 8
// pairs of register-resident operand fragments, no memory traffic in the
// loop. The clock comes from the shader-clock counter (s_memtime) against the
// 100 MHz constant counter (s_memrealtime) over a launch. The power manager
// takes a few launches to settle, so the figure is the fastest of three
// timed launches after a warm-up one.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <vector>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));

constexpr int NT = 512;   // threads per workgroup, one workgroup per CU
constexpr int NF = 8;     // operand fragments of each kind per lane

typedef float f32x4 __attribute__((ext_vector_type(4)));

// SHAPE 0: v_mfma_f32_32x32x16_bf16 (32768 flop); 1: v_mfma_f32_16x16x32_bf16
// (16384 flop, twice as many per trip, so a trip has the same flops).
template <int SHAPE>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
void mfma_ceiling_kernel(const u16x8* src, int iters, float* sink, unsigned long long* clk) {
  const int tid = threadIdx.x;
  unsigned long long t0 = 0, r0 = 0;
  if (blockIdx.x == 0 && tid == 0) {
    t0 = __builtin_amdgcn_s_memtime();
    r0 = __builtin_amdgcn_s_memrealtime();
  }
  bf16x8 a[NF], b[NF];
  const size_t base = ((size_t)blockIdx.x * NT + tid) * (2 * NF);
#pragma unroll
  for (int i = 0; i < NF; ++i) {
    a[i] = __builtin_bit_cast(bf16x8, src[base + i]);
    b[i] = __builtin_bit_cast(bf16x8, src[base + NF + i]);
  }
  float s = 0.f;
  if constexpr (SHAPE == 0) {
    f32x16 acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][e] = 0.f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int j = 0; j < NF; ++j)
#pragma unroll
        for (int i = 0; i < 8; ++i)
          acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(i + j) % NF], b[(i + 2 * j + 1) % NF], acc[i], 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) s += acc[i][e];
  } else {
    f32x4 acc[16];
#pragma unroll
    for (int i = 0; i < 16; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[i][e] = 0.f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int j = 0; j < NF; ++j)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[(i + j) % NF], b[(i + 2 * j + 1) % NF], acc[i], 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < 16; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) s += acc[i][e];
  }
  sink[(size_t)blockIdx.x * NT + tid] = s;   // keeps the products live
  if (blockIdx.x == 0 && tid == 0) {
    clk[0] = __builtin_amdgcn_s_memtime() - t0;
    clk[1] = __builtin_amdgcn_s_memrealtime() - r0;
  }
}

uint16_t to_bf16(float f) {   // round to nearest even
  uint32_t u;
  memcpy(&u, &f, 4);
  return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

// Uniform (0, 1) from a 64-bit counter (splitmix64 finaliser).
double unit(uint64_t x) {
  x += 0x9e3779b97f4a7c15ull;
  x = (x ^ (x >> 30)) * 0xbf58476d1ce4e5b9ull;
  x = (x ^ (x >> 27)) * 0x94d049bb133111ebull;
  x ^= x >> 31;
  return ((double)(x >> 11) + 0.5) * (1.0 / 9007199254740992.0);
}

}  // namespace

extern "C" {

// Runs the MFMA-only kernel on every CU of the current device: shape 0
// v_mfma_f32_32x32x16_bf16, 1 v_mfma_f32_16x16x32_bf16; kind 0 random
// N(0, 1) operands (seeded), 1 all ones, 2 all zeros; `iters` loop trips of
// 64 (shape 0) or 128 (shape 1) MFMAs per wave, the same flops either way.
// After a warm-up launch, three timed launches; writes the fastest one's rate
// in TFLOP/s, its shader clock in MHz and its duration in ms. Allocates and
// frees its own device buffers and synchronises the device. Returns 0, or a
// nonzero hipError_t / -1 for a bad argument.
int malt_calib_mfma_shape(int shape, int kind, int iters, double* tflops, double* clock_mhz, double* ms_out) {
  if (shape < 0 || shape > 1 || kind < 0 || kind > 2 || iters < 1 || !tflops || !clock_mhz || !ms_out) return -1;
  int dev = 0;
  hipDeviceProp_t prop;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipGetDeviceProperties(&prop, dev);
  if (e != hipSuccess) return (int)e;
  const int ncu = prop.multiProcessorCount;
  const size_t nvec = (size_t)ncu * NT * 2 * NF;   // 16-byte operand vectors
  std::vector<uint16_t> h(nvec * 8);
  for (size_t i = 0; i < h.size(); i += 2) {   // Box-Muller pairs
    float v0 = 0.f, v1 = 0.f;
    if (kind == 0) {
      const double u1 = unit(2 * i), u2 = unit(2 * i + 1);
      const double r = sqrt(-2.0 * log(u1));
      v0 = (float)(r * cos(6.283185307179586 * u2));
      v1 = (float)(r * sin(6.283185307179586 * u2));
    } else if (kind == 1) {
      v0 = v1 = 1.f;
    }
    h[i] = to_bf16(v0);
    h[i + 1] = to_bf16(v1);
  }
  u16x8* src = nullptr;
  float* sink = nullptr;
  unsigned long long* clk = nullptr;
  hipEvent_t ev[2] = {nullptr, nullptr};
  e = hipMalloc(&src, nvec * 16);
  if (e == hipSuccess) e = hipMalloc(&sink, (size_t)ncu * NT * sizeof(float));
  if (e == hipSuccess) e = hipMalloc(&clk, 2 * sizeof(unsigned long long));
  if (e == hipSuccess) e = hipMemcpy(src, h.data(), nvec * 16, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipEventCreate(&ev[0]);
  if (e == hipSuccess) e = hipEventCreate(&ev[1]);
  auto kern = shape == 0 ? mfma_ceiling_kernel<0> : mfma_ceiling_kernel<1>;
  const int trip = iters;
  float best = 0.f;
  unsigned long long bc[2] = {0, 0};
  if (e == hipSuccess) {
    hipLaunchKernelGGL(kern, dim3(ncu), dim3(NT), 0, 0, src, trip / 4 + 1, sink, clk);
    for (int rep = 0; rep < 3 && e == hipSuccess; ++rep) {
      float ms = 0.f;
      unsigned long long c[2] = {0, 0};
      e = hipEventRecord(ev[0], 0);
      if (e == hipSuccess) hipLaunchKernelGGL(kern, dim3(ncu), dim3(NT), 0, 0, src, trip, sink, clk);
      if (e == hipSuccess) e = hipGetLastError();
      if (e == hipSuccess) e = hipEventRecord(ev[1], 0);
      if (e == hipSuccess) e = hipEventSynchronize(ev[1]);
      if (e == hipSuccess) e = hipEventElapsedTime(&ms, ev[0], ev[1]);
      if (e == hipSuccess) e = hipMemcpy(c, clk, sizeof(c), hipMemcpyDeviceToHost);
      if (e == hipSuccess && (best == 0.f || ms < best)) {
        best = ms;
        bc[0] = c[0];
        bc[1] = c[1];
      }
    }
  }
  for (hipEvent_t x : ev)
    if (x) (void)hipEventDestroy(x);
  if (clk) (void)hipFree(clk);
  if (sink) (void)hipFree(sink);
  if (src) (void)hipFree(src);
  if (e != hipSuccess) return (int)e;
  const double per_trip = shape == 0 ? NF * 8 * 32768.0 : NF * 16 * 16384.0;
  const double flops = (double)ncu * 8 * (double)trip * per_trip;
  *ms_out = best;
  *tflops = best > 0.f ? flops / (best * 1e-3) / 1e12 : 0.0;
  *clock_mhz = bc[1] ? (double)bc[0] / (double)bc[1] * 100.0 : 0.0;
  return 0;
}

// The 32x32x16 instruction (shape 0) of malt_calib_mfma_shape.
int malt_calib_mfma(int kind, int iters, double* tflops, double* clock_mhz, double* ms_out) {
  return malt_calib_mfma_shape(0, kind, iters, tflops, clock_mhz, ms_out);
}

}  // extern "C"
