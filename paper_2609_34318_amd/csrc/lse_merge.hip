// Exact merge of two ring-step partials of the same rows (ring CP, Sec. 5.2.2):
//   L = M + log(e^(La-M) + e^(Lb-M)), M = max(La, Lb);  O = w_a O_a + w_b O_b,
//   w_x = e^(Lx - L).  Two empty partials (LSE = -inf) stay (0, -inf) with no NaN.
// HBM-bound: 32 lanes per (row, head), each moving 4 fp32 of O_acc and O_part; a capped
// grid strides over the (row, head) pairs.
#include "kernels.h"
#include "prof.h"

namespace hydra {

__global__ __launch_bounds__(256) void lse_merge_kernel(int64_t n_rows, int H, float* __restrict__ o_acc,
                                                        float* __restrict__ lse_acc,
                                                        const float* __restrict__ o_part,
                                                        const float* __restrict__ lse_part,
                                                        uint16_t* __restrict__ o_bf16) {
  const int sub = threadIdx.x & 31;
  const int64_t total = n_rows * H;
  for (int64_t rh = (int64_t)blockIdx.x * 8 + (threadIdx.x >> 5); rh < total; rh += (int64_t)gridDim.x * 8) {
    const int64_t row = rh / H;
    const int head = (int)(rh % H);
    const int64_t li = (int64_t)head * n_rows + row;
    // All 32 lanes of a (row, head) sit in one wave and read lse_acc before lane 0 writes it.
    const float La = lse_acc[li], Lb = lse_part[li];
    const float M = fmaxf(La, Lb);
    float wa = 0.f, wb = 0.f, L = -INFINITY;
    if (M != -INFINITY) {
      const float ea = expf(La - M), eb = expf(Lb - M);
      const float tot = ea + eb;
      L = M + logf(tot);
      wa = ea / tot;
      wb = eb / tot;
    }
    const int64_t off = rh * DV + sub * 4;
    const f32x4 oa = *reinterpret_cast<const f32x4*>(o_acc + off);
    const f32x4 ob = *reinterpret_cast<const f32x4*>(o_part + off);
    f32x4 res;
#pragma unroll
    for (int i = 0; i < 4; ++i) res[i] = (wa > 0.f ? wa * oa[i] : 0.f) + (wb > 0.f ? wb * ob[i] : 0.f);
    *reinterpret_cast<f32x4*>(o_acc + off) = res;
    if (o_bf16) {
      const uint32_t lo = pack_bf16x2(res[0], res[1]), hi = pack_bf16x2(res[2], res[3]);
      *reinterpret_cast<uint2*>(o_bf16 + off) = make_uint2(lo, hi);
    }
    if (sub == 0) lse_acc[li] = L;
  }
}

hipError_t launch_lse_merge(int64_t n_rows, int H, float* o_acc, float* lse_acc, const float* o_part,
                            const float* lse_part, uint16_t* o_bf16, hipStream_t stream) {
  const int64_t blocks = (n_rows * H + 7) / 8 < (1 << 20) ? (n_rows * H + 7) / 8 : (1 << 20);
  const int tok = prof_begin("lse_merge", stream);
  hipLaunchKernelGGL(lse_merge_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, n_rows, H, o_acc, lse_acc,
                     o_part, lse_part, o_bf16);
  prof_end(tok, stream);
  return hipGetLastError();
}

}  // namespace hydra
