// luffy_combine: y[t] = sum over kept slots j of gate[t,j] * y_rep[rep_row[slot_pos[t,j]]]
// One wave per token; 16-byte vector loads and stores (four per lane in
// flight per source row, eight in all); float32 sums.
#include <algorithm>

#include "luffy_common.h"

namespace luffy {
namespace {

// Rows of y_rep are read through a buffer resource: a slot without a
// representative (dropped, or k < 2) and a column chunk past d get the
// out-of-range offset kRange, and robust buffer access returns zeros for
// them.  Every load is therefore unconditional and all of a lane's loads are
// in flight before the first is used (a load behind a branch would wait for
// the one before it).  y_rep must span less than kRange bytes (checked on
// the host against T*k rows).
constexpr uint32_t kRange = 0xFFFF0000u;

// K: slots per token (1 or 2); U: 16-byte chunks per lane per pass (2 when
// two passes' worth of chunks cover a row, else 4), so no load is issued for
// a source or a chunk that cannot exist.
template <bool BF16, int K, int U>
__global__ __launch_bounds__(256) void combine_kernel(const void* __restrict__ y_rep,
                                                      const int32_t* __restrict__ rep_row,
                                                      const int32_t* __restrict__ slot_pos,
                                                      const float* __restrict__ gate, int T, int d,
                                                      void* __restrict__ y) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  constexpr int k = K;
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  constexpr int ES = BF16 ? 2 : 4;          // bytes per element
  constexpr int EPC = 16 / ES;              // elements per 16-byte chunk
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(y_rep),
                                                                       static_cast<short>(0),
                                                                       static_cast<int>(kRange), 0x00020000);
  uint32_t rbase[2] = {kRange, kRange};
  float g[2] = {0.f, 0.f};
  for (int j = 0; j < k; ++j) {
    const int p = slot_pos[static_cast<size_t>(t) * k + j];
    if (p >= 0) {
      rbase[j] = static_cast<uint32_t>(rep_row[p]) * static_cast<uint32_t>(d) * ES;
      g[j] = gate[static_cast<size_t>(t) * k + j];
    }
  }
  // U 16-byte chunks per lane per pass
  for (int c0 = lane * EPC; c0 < d; c0 += U * 64 * EPC) {
    u32x4 v[K][U];
#pragma unroll
    for (int j = 0; j < K; ++j)
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c = c0 + u * 64 * EPC;
        const uint32_t off = (rbase[j] == kRange || c >= d) ? kRange : rbase[j] + static_cast<uint32_t>(c) * ES;
        v[j][u] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
      }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = c0 + u * 64 * EPC;
      if (c >= d) break;
      if constexpr (BF16) {
        float a[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          a[i] = 0.f;
#pragma unroll
          for (int j = 0; j < K; ++j) {
            const uint32_t word = v[j][u][i >> 1];
            const float f = __uint_as_float((i & 1) ? (word & 0xFFFF0000u) : (word << 16));
            a[i] = fmaf(g[j], f, a[i]);
          }
        }
        uint16_t* dst = static_cast<uint16_t*>(y) + static_cast<size_t>(t) * d;
        *reinterpret_cast<uint4*>(dst + c) = make_uint4(pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3]),
                                                        pack_bf16x2(a[4], a[5]), pack_bf16x2(a[6], a[7]));
      } else {
        float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int j = 0; j < K; ++j) {
          a.x = fmaf(g[j], __uint_as_float(v[j][u][0]), a.x);
          a.y = fmaf(g[j], __uint_as_float(v[j][u][1]), a.y);
          a.z = fmaf(g[j], __uint_as_float(v[j][u][2]), a.z);
          a.w = fmaf(g[j], __uint_as_float(v[j][u][3]), a.w);
        }
        float* dst = static_cast<float*>(y) + static_cast<size_t>(t) * d;
        *reinterpret_cast<float4*>(dst + c) = a;
      }
    }
  }
}


// Column-sliced form: the eight XCDs each take one eighth of every row.
// Workgroups are dispatched to the XCDs in turn (block b runs on XCD b % 8),
// so block b covers column slice b % 8 of a run of consecutive tokens, and
// each XCD's L2 only ever holds its slice of y_rep: a representative row
// that several slots use (the condensed duplicates) is fetched from HBM
// about once per slice instead of once per slot.  LPT lanes (a power of two,
// at most 64) share a token's slice, each with CPL 16-byte chunks; a thread
// takes U tokens, tokens_per_pass = 256 / LPT apart, so that U * K * CPL
// loads per lane are in flight before the first is used.
template <bool BF16, int K, int U>
__global__ __launch_bounds__(256) void combine_sliced_kernel(const void* __restrict__ y_rep,
                                                             const int32_t* __restrict__ rep_row,
                                                             const int32_t* __restrict__ slot_pos,
                                                             const float* __restrict__ gate, int T, int d,
                                                             int lpt_log2, int cpl, void* __restrict__ y) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  constexpr int ES = BF16 ? 2 : 4;          // bytes per element
  constexpr int EPC = 16 / ES;              // elements per 16-byte chunk
  const int slice = blockIdx.x & 7;
  const int tb = blockIdx.x >> 3;
  const int lpt = 1 << lpt_log2;
  const int sub = threadIdx.x & (lpt - 1);
  const int tl = threadIdx.x >> lpt_log2;
  const int tpp = 256 >> lpt_log2;          // tokens per pass of the block
  const int slice_chunks = lpt * cpl;
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(y_rep),
                                                                       static_cast<short>(0),
                                                                       static_cast<int>(kRange), 0x00020000);
  int tok[U];
  uint32_t rbase[U][K];
  float g[U][K];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int t = (tb * U + u) * tpp + tl;
    tok[u] = t;
#pragma unroll
    for (int j = 0; j < K; ++j) {
      rbase[u][j] = kRange;
      g[u][j] = 0.f;
      const int p = t < T ? slot_pos[static_cast<size_t>(t) * K + j] : -1;
      if (p >= 0) {
        rbase[u][j] = static_cast<uint32_t>(rep_row[p]) * static_cast<uint32_t>(d) * ES;
        g[u][j] = gate[static_cast<size_t>(t) * K + j];
      }
    }
  }
  for (int cc = 0; cc < cpl; ++cc) {
    const int c = (slice * slice_chunks + cc * lpt + sub) * EPC;   // first element of this lane's chunk
    u32x4 v[U][K];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int j = 0; j < K; ++j) {
        const uint32_t off = rbase[u][j] == kRange ? kRange : rbase[u][j] + static_cast<uint32_t>(c) * ES;
        v[u][j] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
      }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (tok[u] >= T) continue;
      if constexpr (BF16) {
        float a[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          a[i] = 0.f;
#pragma unroll
          for (int j = 0; j < K; ++j) {
            const uint32_t word = v[u][j][i >> 1];
            const float f = __uint_as_float((i & 1) ? (word & 0xFFFF0000u) : (word << 16));
            a[i] = fmaf(g[u][j], f, a[i]);
          }
        }
        uint16_t* dst = static_cast<uint16_t*>(y) + static_cast<size_t>(tok[u]) * d;
        *reinterpret_cast<uint4*>(dst + c) = make_uint4(pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3]),
                                                        pack_bf16x2(a[4], a[5]), pack_bf16x2(a[6], a[7]));
      } else {
        float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int j = 0; j < K; ++j) {
          a.x = fmaf(g[u][j], __uint_as_float(v[u][j][0]), a.x);
          a.y = fmaf(g[u][j], __uint_as_float(v[u][j][1]), a.y);
          a.z = fmaf(g[u][j], __uint_as_float(v[u][j][2]), a.z);
          a.w = fmaf(g[u][j], __uint_as_float(v[u][j][3]), a.w);
        }
        float* dst = static_cast<float*>(y) + static_cast<size_t>(tok[u]) * d;
        *reinterpret_cast<float4*>(dst + c) = a;
      }
    }
  }
}


// ---------------------------------------------------------------- backward
// Transpose of combine (the condensation held fixed): every kept slot adds
// gate * dy[t] to its representative's row, and takes <dy[t], y_rep[r]> as
// its gate gradient.
//
// Row sums through a member list: the kept positions are grouped by
// representative (counts, an exclusive scan, then a fill with one cursor
// per representative; the order inside a group is not fixed), and one wave
// per (representative, 512-column chunk) adds gate * dy[t] of its members
// in registers, four members' rows in flight at a time, and stores the row.

// counts[r] = cursor[r] = 0 for the R rows in use.
__global__ __launch_bounds__(256) void cbwd_clear_kernel(const int32_t* __restrict__ rep_offsets, int E,
                                                         int max_rows, int* __restrict__ cnt,
                                                         int* __restrict__ cursor) {
  const int R = min(rep_offsets[E], max_rows);
  for (int i = blockIdx.x * 256 + threadIdx.x; i < R; i += gridDim.x * 256) {
    cnt[i] = 0;
    cursor[i] = 0;
  }
}

// FILL = false: count the kept positions of each representative;
// FILL = true: place each position in its representative's group.
template <bool FILL>
__global__ __launch_bounds__(256) void cbwd_group_kernel(const int32_t* __restrict__ rep_row,
                                                         const int32_t* __restrict__ offsets, int E, int max_rows,
                                                         int* __restrict__ cnt, const int* __restrict__ start,
                                                         int* __restrict__ cursor, int* __restrict__ list) {
  const int S = offsets[E];
  for (int p = blockIdx.x * 256 + threadIdx.x; p < S; p += gridDim.x * 256) {
    const int r = rep_row[p];
    if (r < 0 || r >= max_rows) continue;
    if constexpr (FILL) list[start[r] + atomicAdd(cursor + r, 1)] = p;
    else atomicAdd(cnt + r, 1);
  }
}

// start[r] = sum of cnt[r'] for r' < r over the R rows in use; one block of
// 1024 threads, each scanning a contiguous run of rows.
__global__ __launch_bounds__(1024) void cbwd_scan_kernel(const int32_t* __restrict__ rep_offsets, int E,
                                                         int max_rows, const int* __restrict__ cnt,
                                                         int* __restrict__ start) {
  __shared__ int part[1024];
  const int R = min(rep_offsets[E], max_rows);
  const int per = (R + 1023) / 1024;
  const int b = threadIdx.x * per, e = min(b + per, R);
  int sum = 0;
  for (int i = b; i < e; ++i) sum += cnt[i];
  part[threadIdx.x] = sum;
  __syncthreads();
  for (int o = 1; o < 1024; o <<= 1) {
    const int v = threadIdx.x >= o ? part[threadIdx.x - o] : 0;
    __syncthreads();
    part[threadIdx.x] += v;
    __syncthreads();
  }
  int run = part[threadIdx.x] - sum;   // exclusive prefix of this thread's run
  for (int i = b; i < e; ++i) {
    start[i] = run;
    run += cnt[i];
  }
  if (threadIdx.x == 1023) start[R] = part[1023];
}

// One wave per (representative r, 512-column chunk): lane l holds columns
// c0 + 8l .. c0 + 8l + 7 (bf16: one 16-byte load per member row; float32:
// two).
template <bool BF16, int K>
__global__ __launch_bounds__(256) void cbwd_rows_kernel(const void* __restrict__ dy,
                                                        const int32_t* __restrict__ perm_token,
                                                        const int32_t* __restrict__ slot_pos,
                                                        const float* __restrict__ gate,
                                                        const int32_t* __restrict__ rep_offsets, int E, int d,
                                                        int max_rows, const int* __restrict__ start,
                                                        const int* __restrict__ list, void* __restrict__ dy_rep) {
  const int lane = threadIdx.x & 63;
  const int R = min(rep_offsets[E], max_rows);
  const int nc = (d + 511) / 512;
  const long long items = static_cast<long long>(R) * nc;
  for (long long it = (static_cast<long long>(blockIdx.x) * 256 + threadIdx.x) >> 6; it < items;
       it += static_cast<long long>(gridDim.x) * 4) {
    const int r = static_cast<int>(it / nc);
    const int c = static_cast<int>(it - static_cast<long long>(r) * nc) * 512 + lane * 8;
    const bool col = c < d;
    const int m0 = start[r], m1 = start[r + 1];
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int m = m0; m < m1; m += 4) {
      int t[4];
      float g[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int mm = min(m + u, m1 - 1);
        const int p = list[mm];
        t[u] = perm_token[p];
        const int j = (K == 2 && slot_pos[static_cast<size_t>(t[u]) * K] != p) ? 1 : 0;
        g[u] = m + u < m1 ? gate[static_cast<size_t>(t[u]) * K + j] : 0.f;
      }
      if (col) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          if constexpr (BF16) {
            const uint4 q = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(dy) +
                                                            static_cast<size_t>(t[u]) * d + c);
            const uint32_t wv[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
            for (int h = 0; h < 4; ++h) {
              acc[2 * h] = fmaf(g[u], __uint_as_float(wv[h] << 16), acc[2 * h]);
              acc[2 * h + 1] = fmaf(g[u], __uint_as_float(wv[h] & 0xFFFF0000u), acc[2 * h + 1]);
            }
          } else {
            const float4* src = reinterpret_cast<const float4*>(static_cast<const float*>(dy) +
                                                                static_cast<size_t>(t[u]) * d + c);
            const float4 a = src[0], b = src[1];
            acc[0] = fmaf(g[u], a.x, acc[0]);
            acc[1] = fmaf(g[u], a.y, acc[1]);
            acc[2] = fmaf(g[u], a.z, acc[2]);
            acc[3] = fmaf(g[u], a.w, acc[3]);
            acc[4] = fmaf(g[u], b.x, acc[4]);
            acc[5] = fmaf(g[u], b.y, acc[5]);
            acc[6] = fmaf(g[u], b.z, acc[6]);
            acc[7] = fmaf(g[u], b.w, acc[7]);
          }
        }
      }
    }
    if (col) {
      if constexpr (BF16) {
        *reinterpret_cast<uint4*>(static_cast<uint16_t*>(dy_rep) + static_cast<size_t>(r) * d + c) =
            make_uint4(pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]), pack_bf16x2(acc[4], acc[5]),
                       pack_bf16x2(acc[6], acc[7]));
      } else {
        float4* dst = reinterpret_cast<float4*>(static_cast<float*>(dy_rep) + static_cast<size_t>(r) * d + c);
        dst[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
        dst[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
      }
    }
  }
}

// Gate gradients: one wave per token, a fixed-order float32 dot product per
// kept slot (0 for a dropped one).
template <bool BF16, int K>
__global__ __launch_bounds__(256) void cbwd_gate_kernel(const void* __restrict__ dy,
                                                        const void* __restrict__ y_rep,
                                                        const int32_t* __restrict__ rep_row,
                                                        const int32_t* __restrict__ slot_pos, int max_rows,
                                                        int T, int d, float* __restrict__ dgate) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  constexpr int EPC = BF16 ? 8 : 4;   // elements per 16-byte chunk
#pragma unroll
  for (int j = 0; j < K; ++j) {
    const int p = slot_pos[static_cast<size_t>(t) * K + j];
    const int r = p >= 0 ? rep_row[p] : -1;
    float dot = 0.f;
    if (r >= 0 && r < max_rows) {
      for (int c = lane * EPC; c < d; c += 64 * EPC) {
        if constexpr (BF16) {
          const uint4 u = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(dy) +
                                                          static_cast<size_t>(t) * d + c);
          const uint4 v = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(y_rep) +
                                                          static_cast<size_t>(r) * d + c);
          const uint32_t uw[4] = {u.x, u.y, u.z, u.w}, vw[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            dot = fmaf(__uint_as_float(uw[i] << 16), __uint_as_float(vw[i] << 16), dot);
            dot = fmaf(__uint_as_float(uw[i] & 0xFFFF0000u), __uint_as_float(vw[i] & 0xFFFF0000u), dot);
          }
        } else {
          const float4 u = *reinterpret_cast<const float4*>(static_cast<const float*>(dy) +
                                                            static_cast<size_t>(t) * d + c);
          const float4 v = *reinterpret_cast<const float4*>(static_cast<const float*>(y_rep) +
                                                            static_cast<size_t>(r) * d + c);
          dot = fmaf(u.x, v.x, dot);
          dot = fmaf(u.y, v.y, dot);
          dot = fmaf(u.z, v.z, dot);
          dot = fmaf(u.w, v.w, dot);
        }
      }
    }
    // fixed-order butterfly: every lane holds the same sum
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) dot += __shfl_xor(dot, o, 64);
    if (lane == 0) dgate[static_cast<size_t>(t) * K + j] = dot;
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
  if (static_cast<double>(T) * k * d * (dtype == LUFFY_BF16 ? 2 : 4) >= static_cast<double>(kRange))
    return fail(LUFFY_E_UNSUPPORTED, "luffy_combine: y_rep of up to T*k=%lld rows of d=%d must span < 4 GiB - 64 KiB",
                static_cast<long long>(T) * k, d);
  hipStream_t s = static_cast<hipStream_t>(stream);
  // Top-2 (two source rows a token) takes the column-sliced kernel when a
  // row's 16-byte chunks split into eight slices of 2^n (n <= 6) or of a
  // multiple of 64 chunks; top-1, or other widths, one wave per token.
  // Measured on the expert-parallel share (T = 32768, d = 2048, top-2):
  // HBM reads 252 -> 136 MB and 57.7 -> 53.3 us; on a top-1 layer of
  // 65536 tokens (d = 1024) the sliced form ran 30.5 -> 32.5 us.
  const int chunks = d * (dtype == LUFFY_BF16 ? 2 : 4) / 16;
  const int sc = chunks / 8;
  if (k == 2 && chunks % 8 == 0 && ((sc & (sc - 1)) == 0 || sc % 64 == 0)) {
    const int lpt = std::min(sc, 64);
    const int lpt_log2 = __builtin_ctz(static_cast<unsigned>(lpt));
    const int cpl = sc / lpt;
    const long long tok_per_block = static_cast<long long>(256 / lpt) * 4;
    const int sblocks = static_cast<int>(8 * ((T + tok_per_block - 1) / tok_per_block));
#define LUFFY_COMBINE_S(BF, K_, U_) launch("combine", combine_sliced_kernel<BF, K_, U_>, sblocks, 256, 0, s, y_rep, \
                                           rep_row, slot_pos, topk_gate, T, d, lpt_log2, cpl, y)
    if (dtype == LUFFY_BF16) LUFFY_COMBINE_S(true, 2, 4);
    else LUFFY_COMBINE_S(false, 2, 4);
#undef LUFFY_COMBINE_S
    return check_launch("luffy_combine");
  }
  const int blocks = (T + 3) / 4;
  const bool two = d * (dtype == LUFFY_BF16 ? 2 : 4) <= 2 * 64 * 16;   // two chunks per lane cover a row
#define LUFFY_COMBINE(BF, K_, U_) launch("combine", combine_kernel<BF, K_, U_>, blocks, 256, 0, s, y_rep, rep_row, \
                                         slot_pos, topk_gate, T, d, y)
  if (dtype == LUFFY_BF16) {
    if (k == 1) { if (two) LUFFY_COMBINE(true, 1, 2); else LUFFY_COMBINE(true, 1, 4); }
    else { if (two) LUFFY_COMBINE(true, 2, 2); else LUFFY_COMBINE(true, 2, 4); }
  } else {
    if (k == 1) { if (two) LUFFY_COMBINE(false, 1, 2); else LUFFY_COMBINE(false, 1, 4); }
    else { if (two) LUFFY_COMBINE(false, 2, 2); else LUFFY_COMBINE(false, 2, 4); }
  }
#undef LUFFY_COMBINE
  return check_launch("luffy_combine");
}

struct CbwdWs {
  int *cnt, *start, *cursor, *list;
};

CbwdWs carve_cbwd(Carver& c, int max_rows, long long slots) {
  CbwdWs w;
  w.cnt = c.take<int>(static_cast<size_t>(max_rows));
  w.start = c.take<int>(static_cast<size_t>(max_rows) + 1);
  w.cursor = c.take<int>(static_cast<size_t>(max_rows));
  w.list = c.take<int>(static_cast<size_t>(slots));
  return w;
}

extern "C" size_t luffy_combine_backward_workspace_size(int T, int k, int max_rows) {
  if (T <= 0 || k <= 0 || max_rows <= 0) return 0;
  Carver c(nullptr);
  carve_cbwd(c, max_rows, static_cast<long long>(T) * k);
  return c.size();
}

extern "C" int luffy_combine_backward(const void* dy, const void* y_rep, const int32_t* rep_row,
                                      const int32_t* perm_token, const int32_t* slot_pos,
                                      const float* topk_gate, const int32_t* offsets,
                                      const int32_t* rep_offsets, int E, int T, int k, int d, int dtype,
                                      int max_rows, void* dy_rep, float* dgate, void* workspace,
                                      size_t workspace_bytes, void* stream) {
  if (!dy || !y_rep || !rep_row || !perm_token || !slot_pos || !topk_gate || !offsets || !rep_offsets ||
      !dy_rep || !dgate)
    return fail(LUFFY_E_INVALID, "luffy_combine_backward: null pointer argument");
  if (T <= 0 || d <= 0 || E <= 0 || max_rows <= 0)
    return fail(LUFFY_E_INVALID, "luffy_combine_backward: T=%d d=%d E=%d max_rows=%d", T, d, E, max_rows);
  if (k != 1 && k != 2) return fail(LUFFY_E_INVALID, "luffy_combine_backward: k=%d must be 1 or 2", k);
  if (dtype != LUFFY_F32 && dtype != LUFFY_BF16)
    return fail(LUFFY_E_INVALID, "luffy_combine_backward: unknown dtype %d", dtype);
  if (d % 64 != 0) return fail(LUFFY_E_UNSUPPORTED, "luffy_combine_backward: d=%d not a multiple of 64", d);
  if (static_cast<long long>(T) * k >= (1ll << 31))
    return fail(LUFFY_E_UNSUPPORTED, "luffy_combine_backward: T*k >= 2^31");
  const size_t need = luffy_combine_backward_workspace_size(T, k, max_rows);
  if (workspace_bytes < need || !workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u))
    return fail(LUFFY_E_WORKSPACE, "luffy_combine_backward: workspace needs %zu bytes, 256-aligned", need);
  hipStream_t s = static_cast<hipStream_t>(stream);
  Carver c(workspace);
  const CbwdWs ws = carve_cbwd(c, max_rows, static_cast<long long>(T) * k);
  const int S = T * k;
  const int rblocks = std::max(1, std::min((max_rows + 255) / 256, 1024));
  const int sblocks = std::max(1, std::min((S + 255) / 256, 2048));
  launch("cbwd_group", cbwd_clear_kernel, rblocks, 256, 0, s, rep_offsets, E, max_rows, ws.cnt, ws.cursor);
  launch("cbwd_group", cbwd_group_kernel<false>, sblocks, 256, 0, s, rep_row, offsets, E, max_rows, ws.cnt,
         static_cast<const int*>(ws.start), ws.cursor, ws.list);
  launch("cbwd_group", cbwd_scan_kernel, 1, 1024, 0, s, rep_offsets, E, max_rows, static_cast<const int*>(ws.cnt),
         ws.start);
  launch("cbwd_group", cbwd_group_kernel<true>, sblocks, 256, 0, s, rep_row, offsets, E, max_rows, ws.cnt,
         static_cast<const int*>(ws.start), ws.cursor, ws.list);
  const long long row_waves = static_cast<long long>(max_rows) * ((d + 511) / 512);
  const int row_blocks = static_cast<int>(std::max(1ll, std::min((row_waves + 3) / 4, 8192ll)));
  const int blocks = (T + 3) / 4;
#define LUFFY_CBWD(BF, K_)                                                                                     \
  do {                                                                                                         \
    launch("cbwd_rows", cbwd_rows_kernel<BF, K_>, row_blocks, 256, 0, s, dy, perm_token, slot_pos, topk_gate,  \
           rep_offsets, E, d, max_rows, static_cast<const int*>(ws.start), static_cast<const int*>(ws.list),   \
           dy_rep);                                                                                            \
    launch("cbwd_gate", cbwd_gate_kernel<BF, K_>, blocks, 256, 0, s, dy, y_rep, rep_row, slot_pos, max_rows,   \
           T, d, dgate);                                                                                       \
  } while (0)
  if (dtype == LUFFY_BF16) { if (k == 1) LUFFY_CBWD(true, 1); else LUFFY_CBWD(true, 2); }
  else { if (k == 1) LUFFY_CBWD(false, 1); else LUFFY_CBWD(false, 2); }
#undef LUFFY_CBWD
  return check_launch("luffy_combine_backward");
}

