// Internal declarations shared by the libkvec translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "kvec.h"

namespace kvec {

constexpr int kWave = 64;

// Key-tile sizes of the two window-score passes (multiples of 16).
constexpr int kTilePass1 = 512;
constexpr int kTilePass2 = 256;
// Tokens per block of the pooling/statistics kernel.
constexpr int kPoolBlock = 256;
// Threads of the per-head selection kernels.
constexpr int kSelectThreads = 1024;

// Derived geometry of one problem.
struct Geometry {
  int batch, layers, H, HQ, G, D, T, O, Wn, Tc, B, pool, delta;
  float lam, beta;
  int dtype;
  int Kp;        // preserved tokens per head
  int M;         // prefix picks per head, B - O
  int RB;        // 16-row window blocks per row tile
  int WR;        // window rows per row tile, 16 * RB
  int n_rt;      // row tiles covering the Wn window rows
  int n_rt_base; // row tiles (from the newest) holding base-window rows
  int n_kt1;     // key tiles of pass 1 over [0, T)
  int n_kt2;     // key tiles of pass 2 over [0, Tc)
  int SK;        // keys per importance exchange in pass 2
  int n_pool_blk;
  int words;     // ceil(T / 64)
  int esize;     // bytes per element of Q/K/V
  bool keep_all; // T <= B
};

// Workspace carve-up (byte offsets, each 256-byte aligned).
struct Workspace {
  size_t lse_part;   // float2 [batch][HQ][Wn][n_kt1]
  size_t lse2;       // float  [batch][HQ][Wn]
  size_t psum_base;  // float  [batch][n_rt][H][Tc]
  size_t psum_all;   // float  [batch][n_rt][H][Tc]
  size_t ipart;      // float  [batch][n_rt][Tc]
  size_t p_raw;      // float  [batch][H][Tc]   (evict paths only)
  size_t p_ext;      // float  [batch][H][Tc]
  size_t imp;        // float  [batch][Tc]
  size_t pooled;     // float  [batch][H][Tc]
  size_t pooled_ext; // float  [batch][H][Tc]
  size_t stats;      // double2 [batch][H][n_pool_blk]
  size_t use_ext;    // int32  [batch][H]
  size_t keep;       // uint32 [batch][H][ceil(Tc/32)]
  size_t keys;       // uint32 [batch][H][Tc]
  size_t total;
};

kvec_status make_geometry(const kvec_config* cfg, Geometry* g);
Workspace make_workspace(const Geometry& g);

// Launchers (return hipSuccess or the launch error).
hipError_t launch_score(const Geometry& g, const void* q, const int64_t qs[3], const void* k,
                        const int64_t ks[3], float* p_raw, float* p_ext, float* imp, char* ws,
                        const Workspace& w, hipStream_t s, hipEvent_t* ev);
hipError_t launch_select(const Geometry& g, int layer, const float* p_raw, const float* p_ext,
                         const float* imp, uint64_t* bits, int32_t* idx, uint32_t* htop_mask,
                         char* ws, const Workspace& w, hipStream_t s);
hipError_t launch_keep_all(const Geometry& g, int layer, uint64_t* bits, int32_t* idx,
                           hipStream_t s);
hipError_t launch_compact(const Geometry& g, int n_layers, const void* k, const int64_t ks[4],
                          const void* v, const int64_t vs[4], const int32_t* idx, void* k_out,
                          void* v_out, hipStream_t s);
hipError_t launch_coverage(const Geometry& g, const uint64_t* bits, int upto, int64_t* count,
                           hipStream_t s);
hipError_t launch_zero_bits(const Geometry& g, uint64_t* bits, hipStream_t s);

// ---------------------------------------------------------------------------
// Device helpers
// ---------------------------------------------------------------------------

// Order-preserving map of an IEEE float to uint32 (larger float -> larger key).
__device__ __forceinline__ uint32_t float_key(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ int wave_incl_scan(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(v, o);
    if (lane >= o) v += u;
  }
  return v;
}

// Exclusive prefix sum over the whole work-group (blockDim.x a multiple of 64,
// at most 1024).  `tmp` is >= 17 ints of shared memory.  Returns the
// exclusive prefix; `total` receives the block sum.  Contains barriers.
__device__ __forceinline__ int block_excl_scan(int v, int* tmp, int& total) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  const int incl = wave_incl_scan(v);
  if (lane == 63) tmp[wid] = incl;
  __syncthreads();
  if (wid == 0) {
    const int x = lane < nw ? tmp[lane] : 0;
    const int xi = wave_incl_scan(x);
    if (lane < nw) tmp[lane] = xi - x;
    if (lane == nw - 1) tmp[16] = xi;
  }
  __syncthreads();
  const int r = tmp[wid] + incl - v;
  total = tmp[16];
  __syncthreads();
  return r;
}

}  // namespace kvec
