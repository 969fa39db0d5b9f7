// luffy_combine: y[t] = sum over kept slots j of gate[t,j] * y_rep[rep_row[slot_pos[t,j]]]
// One wave per token; 16-byte vector loads and stores (four per lane in
// flight per source row); float32 sums.
#include "luffy_common.h"

namespace luffy {
namespace {

template <bool BF16>
__global__ __launch_bounds__(256) void combine_kernel(const void* __restrict__ y_rep,
                                                      const int32_t* __restrict__ rep_row,
                                                      const int32_t* __restrict__ slot_pos,
                                                      const float* __restrict__ gate, int T, int k,
                                                      int d, void* __restrict__ y) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  int row[2] = {-1, -1};
  float g[2] = {0.f, 0.f};
  for (int j = 0; j < k; ++j) {
    const int p = slot_pos[static_cast<size_t>(t) * k + j];
    if (p >= 0) {
      row[j] = rep_row[p];
      g[j] = gate[static_cast<size_t>(t) * k + j];
    }
  }
  // four 16-byte chunks per lane per pass, all loads issued before use
  if constexpr (BF16) {
    const uint16_t* src = static_cast<const uint16_t*>(y_rep);
    uint16_t* dst = static_cast<uint16_t*>(y) + static_cast<size_t>(t) * d;
    for (int c0 = lane * 8; c0 < d; c0 += 4 * 512) {
      Pack16 v[2][4];
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int c = c0 + u * 512;
          if (j < k && row[j] >= 0 && c < d)
            v[j][u].u4 = *reinterpret_cast<const uint4*>(src + static_cast<size_t>(row[j]) * d + c);
          else
            v[j][u].u4 = make_uint4(0, 0, 0, 0);
        }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = c0 + u * 512;
        if (c >= d) break;
        float a[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          a[i] = 0.f;
#pragma unroll
          for (int j = 0; j < 2; ++j) a[i] = fmaf(g[j], bf16_to_f32(v[j][u].h[i]), a[i]);
        }
        *reinterpret_cast<uint4*>(dst + c) = make_uint4(pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3]),
                                                        pack_bf16x2(a[4], a[5]), pack_bf16x2(a[6], a[7]));
      }
    }
  } else {
    const float* src = static_cast<const float*>(y_rep);
    float* dst = static_cast<float*>(y) + static_cast<size_t>(t) * d;
    for (int c0 = lane * 4; c0 < d; c0 += 4 * 256) {
      float4 v[2][4];
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int c = c0 + u * 256;
          if (j < k && row[j] >= 0 && c < d)
            v[j][u] = *reinterpret_cast<const float4*>(src + static_cast<size_t>(row[j]) * d + c);
          else
            v[j][u] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = c0 + u * 256;
        if (c >= d) break;
        float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          a.x = fmaf(g[j], v[j][u].x, a.x);
          a.y = fmaf(g[j], v[j][u].y, a.y);
          a.z = fmaf(g[j], v[j][u].z, a.z);
          a.w = fmaf(g[j], v[j][u].w, a.w);
        }
        *reinterpret_cast<float4*>(dst + c) = a;
      }
    }
  }
}

}  // namespace
}  // namespace luffy

using namespace luffy;

extern "C" int luffy_combine(const void* y_rep, const int32_t* rep_row,
                             const int32_t* slot_pos, const float* topk_gate,
                             int T, int k, int d, int dtype, void* y, void* stream) {
  if (!y_rep || !rep_row || !slot_pos || !topk_gate || !y)
    return fail(LUFFY_E_INVALID, "luffy_combine: null pointer argument");
  if (T <= 0 || d <= 0) return fail(LUFFY_E_INVALID, "luffy_combine: T=%d d=%d", T, d);
  if (k != 1 && k != 2) return fail(LUFFY_E_INVALID, "luffy_combine: k=%d must be 1 or 2", k);
  if (dtype != LUFFY_F32 && dtype != LUFFY_BF16)
    return fail(LUFFY_E_INVALID, "luffy_combine: unknown dtype %d", dtype);
  if (d % 64 != 0) return fail(LUFFY_E_UNSUPPORTED, "luffy_combine: d=%d not a multiple of 64", d);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int blocks = (T + 3) / 4;
  if (dtype == LUFFY_BF16)
    launch("combine", combine_kernel<true>, blocks, 256, 0, s, y_rep, rep_row, slot_pos, topk_gate, T, k, d, y);
  else
    launch("combine", combine_kernel<false>, blocks, 256, 0, s, y_rep, rep_row, slot_pos, topk_gate, T, k, d, y);
  return check_launch("luffy_combine");
}
