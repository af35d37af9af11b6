// Debug entry point: the per-token quantities of one chunk's inner gradient
// for one (batch row, head) chain, every token at the same weights W (the
// chunkwise rule of Sec. 2.2; the chain rule of the recall loss of Sec. 2.1):
//   Zk = K W1^T (C x hid),  R = (2/d) (s(Zk) W2^T - V) (C x d),
//   D1 = (R W2) * s'(Zk) (C x hid),
// so that token t's gradients are u1_t = D1_t^T k_t and u2_t = R_t^T s(Zk_t).
// One workgroup, fp32 arithmetic on the I/O-dtype keys and values, the
// activation and its derivative from the same device routines as the layer.
#include "tnt_device.h"
#include "tnt_kernels.h"

namespace tnt {

template <typename IO, int ACT>
__global__ void __launch_bounds__(256) dbg_chunk_grads_kernel(DbgArgs a) {
  const int d = a.d, hid = a.hid, C = a.C;
  const IO* k = (const IO*)a.k + a.tok0 * d;
  const IO* v = (const IO*)a.v + a.tok0 * d;
  for (int e = threadIdx.x; e < C * hid; e += blockDim.x) {  // Zk = K W1^T
    const int i = e / hid, j = e - i * hid;
    float s = 0.f;
    for (int l = 0; l < d; ++l) s += to_f(k[(size_t)i * d + l]) * a.W1[(size_t)j * d + l];
    a.Zk[e] = s;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < C * d; e += blockDim.x) {  // R = (2/d)(s(Zk) W2^T - V)
    const int i = e / d, m = e - i * d;
    float s = 0.f;
    for (int j = 0; j < hid; ++j) s += act_f<ACT>(a.Zk[(size_t)i * hid + j]) * a.W2[(size_t)m * hid + j];
    a.R[e] = (2.0f / (float)d) * (s - to_f(v[(size_t)i * d + m]));
  }
  __syncthreads();
  for (int e = threadIdx.x; e < C * hid; e += blockDim.x) {  // D1 = (R W2) * s'(Zk)
    const int i = e / hid, j = e - i * hid;
    float s = 0.f;
    for (int m = 0; m < d; ++m) s += a.R[(size_t)i * d + m] * a.W2[(size_t)m * hid + j];
    a.D1[e] = s * act_all<ACT>(a.Zk[e]).d1;
  }
}

hipError_t launch_dbg_chunk_grads(const DbgArgs& a, hipStream_t st) {
  if (a.bf16) {
    if (a.act == ACT_SILU)
      hipLaunchKernelGGL((dbg_chunk_grads_kernel<__bf16, ACT_SILU>), dim3(1), dim3(256), 0, st, a);
    else
      hipLaunchKernelGGL((dbg_chunk_grads_kernel<__bf16, ACT_GELU>), dim3(1), dim3(256), 0, st, a);
  } else {
    if (a.act == ACT_SILU)
      hipLaunchKernelGGL((dbg_chunk_grads_kernel<float, ACT_SILU>), dim3(1), dim3(256), 0, st, a);
    else
      hipLaunchKernelGGL((dbg_chunk_grads_kernel<float, ACT_GELU>), dim3(1), dim3(256), 0, st, a);
  }
  return hipGetLastError();
}

}  // namespace tnt
