// Cache store of the kept tokens (paper Sec. 4.1: the K/V of the selected
// tokens is stored for decoding).  A byte copy: each thread moves one 16-byte
// chunk of a K row and the same chunk of the V row, so consecutive threads
// write consecutive bytes of the compacted [.., B, d] cache and read
// consecutive bytes within a source row.
#include "kvec_internal.h"

namespace kvec {
namespace {

struct GatherArgs {
  const char* k;
  const char* v;
  int64_t ks_l, ks_b, ks_h, ks_t;  // element strides
  int64_t vs_l, vs_b, vs_h, vs_t;
  const int32_t* idx;              // [L][batch][H][B]
  char* k_out;
  char* v_out;
  int batch, H, B, T, chunks, esize;
};

__global__ void gather_kernel(GatherArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int b = blockIdx.y, l = blockIdx.z;
  const int64_t per_seq = (int64_t)a.H * a.B * a.chunks;
  if (i >= per_seq) return;
  const int ch = (int)(i % a.chunks);
  const int64_t rowi = i / a.chunks;  // h * B + slot
  const int h = (int)(rowi / a.B);
  const int64_t orow = ((int64_t)l * a.batch + b) * a.H * a.B + rowi;
  const int id = a.idx[orow];
  const int64_t rb = (int64_t)a.chunks * 16;
  uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
  if (id >= 0 && id < a.T) {
    const int64_t ko = ((int64_t)l * a.ks_l + (int64_t)b * a.ks_b + (int64_t)h * a.ks_h +
                        (int64_t)id * a.ks_t) * a.esize;
    const int64_t vo = ((int64_t)l * a.vs_l + (int64_t)b * a.vs_b + (int64_t)h * a.vs_h +
                        (int64_t)id * a.vs_t) * a.esize;
    kv = reinterpret_cast<const uint4*>(a.k + ko)[ch];
    vv = reinterpret_cast<const uint4*>(a.v + vo)[ch];
  }
  reinterpret_cast<uint4*>(a.k_out + orow * rb)[ch] = kv;
  reinterpret_cast<uint4*>(a.v_out + orow * rb)[ch] = vv;
}

}  // namespace

hipError_t launch_compact(const Geometry& g, int n_layers, const void* k, const int64_t ks[4],
                          const void* v, const int64_t vs[4], const int32_t* idx, void* k_out,
                          void* v_out, hipStream_t s) {
  GatherArgs a;
  a.k = static_cast<const char*>(k);
  a.v = static_cast<const char*>(v);
  a.ks_l = ks[0]; a.ks_b = ks[1]; a.ks_h = ks[2]; a.ks_t = ks[3];
  a.vs_l = vs[0]; a.vs_b = vs[1]; a.vs_h = vs[2]; a.vs_t = vs[3];
  a.idx = idx;
  a.k_out = static_cast<char*>(k_out);
  a.v_out = static_cast<char*>(v_out);
  a.batch = g.batch;
  a.H = g.H;
  a.B = g.B;
  a.T = g.T;
  a.esize = g.esize;
  a.chunks = g.D * g.esize / 16;
  const int64_t per_seq = (int64_t)g.H * g.B * a.chunks;
  hipLaunchKernelGGL(gather_kernel, dim3((unsigned)((per_seq + 255) / 256), g.batch, n_layers),
                     dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace kvec
