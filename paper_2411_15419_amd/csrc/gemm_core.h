// Output tile of C[i][j] = sum_k P[i][k] * Q[j][k] on bf16 MFMA (gfx950).
//
// Both operands are row-major with the contraction index contiguous, so one
// core serves the similarity tiles (P and Q are gathered token rows of one
// bucket) and the FFN tiles (P = weight rows in [out, in] layout, Q =
// gathered token rows).
//
// Block tile 256 x 256; waves form a WM x WN grid, each owning a
// (256/WM) x (256/WN) sub-tile of v_mfma_f32_32x32x16_bf16 blocks.  Waves
// are dealt to the four SIMDs of a CU round-robin (wave w on SIMD w % 4).
// With MFAST the wave's P-block index varies fastest (wm = w % WM), so with
// WM = 4 every SIMD holds one P quarter and every Q part: a tile whose Q
// rows are only partly valid can skip the MFMAs of its invalid 32-row Q
// blocks (run<NQ>) and still keep the four SIMDs equally loaded.
//
// K advances 32 at a time through a ring of 4 LDS stages (32 KB each).
// Operands go from global memory straight into LDS with buffer loads
// (buffer_load_dwordx4 ... lds, no staging registers; 32-bit byte offsets
// from a buffer resource, so each operand must span less than 4 GiB):
// while stage kt is multiplied from registers, stage kt+1 is read out of
// LDS and stages kt+2..kt+4 are in flight.  In the steady state the
// multiplies of a stage are interleaved one-to-one with the buffer loads
// and LDS reads of later stages.  LDS rows are 64 bytes with no padding; the four
// 16-byte chunks of row r are stored XOR-permuted by (r>>2) & 3, so the 16
// lanes the LDS serves together in a fragment read (16 consecutive rows, one
// chunk) hit 16 distinct 16-byte bank groups, while each DMA instruction
// still writes one contiguous 1 KB block.
//
// Operand rows are given as 32-bit element offsets from a base pointer
// (every operand here has fewer than 2^31 elements).
//
// Result layout of acc[fm][fn][v] in lane l of wave w:
//   P row  wave_m(w) * WTM + 32*fm + 8*(v/4) + 4*(l/32) + v%4
//   Q row  wave_n(w) * WTN + 32*fn + l%32
#pragma once

#include "luffy_common.h"

namespace luffy {

typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;

__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Workgroup barrier without the memory fences of __syncthreads(): the fence
// would make the compiler wait for every outstanding DMA load.  LDS
// visibility is handled explicitly: each wave waits (vmcnt) for its own DMA
// writes before the barrier, and LDS reads are issued after it.
__device__ __forceinline__ void raw_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// s_waitcnt with only the vector-memory counter constrained (<= N, N < 64;
// the 6-bit count is split over bits 3:0 and 15:14).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | (0x7 << 4) | (0xF << 8) | ((N >> 4) << 14));
}

template <int WM_, int WN_, bool MFAST_ = false>
struct Gemm256 {
  static constexpr int BM = 256, BN = 256, WM = WM_, WN = WN_;
  static constexpr int BK = 32;                      // K per stage
  static constexpr int STAGES = 4;
  static constexpr int THREADS = 64 * WM * WN;       // 512
  static constexpr int WTM = BM / WM, WTN = BN / WN; // 128 x 64
  static constexpr int FM = WTM / 32, FN = WTN / 32; // 4 x 2
  static constexpr int ROW_BYTES = BK * 2;           // 64
  static constexpr int STAGE_BYTES = (BM + BN) * ROW_BYTES;   // 32 KB
  static constexpr int LDS_BYTES = STAGES * STAGE_BYTES;      // 128 KB
  // each wave instruction fills 16 rows (1 KB); 32 per stage
  static constexpr int NWAVES = WM * WN;
  static constexpr int LOADS = (BM + BN) / 16 / NWAVES;
  static_assert(LOADS * NWAVES * 16 == BM + BN && LOADS % 2 == 0, "load plan");

  using Acc = f32x16[FM][FN];

  static __device__ __forceinline__ int swz(int r) { return (r >> 2) & 3; }

  // wave -> (P block, Q block) of the wave grid
  static __device__ __forceinline__ int wave_m(int w) { return MFAST_ ? w % WM : w / WN; }
  static __device__ __forceinline__ int wave_n(int w) { return MFAST_ ? w / WM : w % WN; }

  // Stage row this lane fills in load j: P rows 0..255 then Q rows 256..511
  // (loads 0 .. LOADS/2-1 fill P rows, the rest Q rows).
  static __device__ __forceinline__ int wave() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

  static __device__ __forceinline__ int load_row(int j) {
    const int w = wave(), lane = threadIdx.x & 63;
    return (w + NWAVES * j) * 16 + (lane >> 2);
  }

  static __device__ __forceinline__ void zero(Acc& acc) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
  }

  // Issue the DMA of K slice [k0, k0+32) into stage buffer `st`.
  // goff[j]: byte offset of the row load_row(j) (rows 0..255 from the P
  // resource, 256..511 from the Q resource), already including this lane's
  // XOR-permuted chunk.  w: wave index (wave-uniform).
  using lds_ptr = __attribute__((address_space(3))) uint8_t*;

  static __device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base) {
    // raw buffer (no stride), full 32-bit range; 0x00020000: gfx9 word 3
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0),
                                             static_cast<int>(0xFFFFFFFFu), 0x00020000);
  }

  static __device__ __forceinline__ void issue(__amdgpu_buffer_rsrc_t prs, __amdgpu_buffer_rsrc_t qrs,
                                               const uint32_t (&goff)[LOADS], int k0, lds_ptr st,
                                               int w) {
#pragma unroll
    for (int j = 0; j < LOADS; ++j) {
      lds_ptr dst = st + (w + NWAVES * j) * 16 * ROW_BYTES;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(j < LOADS / 2 ? prs : qrs,
                                               reinterpret_cast<__attribute__((address_space(3))) void*>(dst),
                                               16, goff[j], k0 * 2, 0, 0);
    }
  }

  struct Frags {
    bf16x8 a[2][FM], b[2][FN];
  };

  // LDS -> registers: both 16-wide substeps of one stage, for the first NQ
  // of the wave's FN Q blocks (none at all when NQ = 0).
  template <int NQ = FN>
  static __device__ __forceinline__ void read_frags(lds_ptr S, int prow0, int qrow0, int half, int sw,
                                                    Frags& f) {
    if constexpr (NQ > 0) {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const int pc = ((2 * kk + half) ^ sw) * 16;
#pragma unroll
        for (int i = 0; i < FM; ++i)
          f.a[kk][i] = *reinterpret_cast<const __attribute__((address_space(3))) bf16x8*>(
              S + prow0 + 32 * i * ROW_BYTES + pc);
#pragma unroll
        for (int j = 0; j < NQ; ++j)
          f.b[kk][j] = *reinterpret_cast<const __attribute__((address_space(3))) bf16x8*>(
              S + qrow0 + 32 * j * ROW_BYTES + pc);
      }
    }
  }

  template <int NQ = FN>
  static __device__ __forceinline__ void mma(const Frags& f, Acc& acc) {
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < NQ; ++j) acc[i][j] = mfma32x32x16(f.a[kk][i], f.b[kk][j], acc[i][j]);
  }

  // DMA: lane fills physical chunk lane%4 of its row with logical chunk
  // (lane%4) ^ swz(row); byte offsets.
  static __device__ __forceinline__ void dma_offsets(const uint32_t (&poff)[LOADS / 2],
                                                     const uint32_t (&qoff)[LOADS / 2],
                                                     uint32_t (&goff)[LOADS]) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int j = 0; j < LOADS; ++j) {
      const int r = load_row(j);
      const uint32_t lc = static_cast<uint32_t>((lane & 3) ^ swz(r));
      goff[j] = ((j < LOADS / 2 ? poff[j] : qoff[j - LOADS / 2]) + lc * 8) * 2u;
    }
  }

  // Scheduling of one steady-state stage: each MFMA is followed by one of
  // the stage's buffer loads, then by one LDS read, until they run out;
  // loads and reads left over (few Q blocks) follow the last MFMA.
  template <int NQ = FN>
  static __device__ __forceinline__ void interleave() {
    constexpr int NMF = FM * NQ * 2, NDS = NQ > 0 ? (FM + NQ) * 2 : 0, NVM = LOADS;
    constexpr int PV = NMF < NVM ? NMF : NVM;
    constexpr int PD = (NMF - PV) < NDS ? (NMF - PV) : NDS;
#pragma unroll
    for (int i = 0; i < PV; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // VMEM read
    }
#pragma unroll
    for (int i = 0; i < PD; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // DS read
    }
    if constexpr (NMF > PV + PD) __builtin_amdgcn_sched_group_barrier(0x008, NMF - PV - PD, 0);
    if constexpr (NVM > PV) __builtin_amdgcn_sched_group_barrier(0x020, NVM - PV, 0);
    if constexpr (NDS > PD) __builtin_amdgcn_sched_group_barrier(0x100, NDS - PD, 0);
  }

  // Wait until the DMA of a stage has landed in this wave while the loads of
  // `later` (0..3) stages issued after it stay in flight.
  static __device__ __forceinline__ void wait_stage(int later) {
    if (later >= 3) wait_vmcnt<3 * LOADS>();
    else if (later == 2) wait_vmcnt<2 * LOADS>();
    else if (later == 1) wait_vmcnt<LOADS>();
    else wait_vmcnt<0>();
  }

  // poff[j] (j < LOADS/2): element offset of P row load_row(j);
  // qoff[j] (j < LOADS/2): element offset of Q row load_row(j + LOADS/2) - 256.
  // K must be a multiple of 32.  Ends with a barrier after which the LDS may
  // be reused.  NQ: the wave multiplies only its first NQ Q blocks (the
  // accumulators of the others stay as they are); every wave still loads
  // its share of the operands and takes every barrier, whatever its NQ.
  //
  // Iteration kt: wait for stage kt+1 (DMA) and for this wave's reads of
  // stage kt, barrier, issue the DMA of stage kt+4 into stage kt's buffer,
  // request stage kt+1's fragments, then multiply stage kt from registers,
  // so the LDS reads of one stage overlap the MFMAs of the previous one.
  template <int NQ = FN>
  static __device__ __forceinline__ void run(const uint16_t* __restrict__ pbase,
                                             const uint32_t (&poff)[LOADS / 2],
                                             const uint16_t* __restrict__ qbase,
                                             const uint32_t (&qoff)[LOADS / 2], int K,
                                             uint8_t* lds_generic, Acc& acc) {
    const lds_ptr lds = (lds_ptr)lds_generic;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = wave();
    const int wm = wave_m(w), wn = wave_n(w);
    const __amdgpu_buffer_rsrc_t prs = rsrc(pbase), qrs = rsrc(qbase);
    uint32_t goff[LOADS];
    dma_offsets(poff, qoff, goff);
    const int nk = K / BK;
#pragma unroll
    for (int st = 0; st < STAGES; ++st)
      if (st < nk) issue(prs, qrs, goff, st * BK, lds + st * STAGE_BYTES, w);

    // fragment reads: lane reads row (l%32) of each 32-row block, logical
    // chunk kk/8 + l/32
    const int sw = swz(lane & 31);
    const int prow0 = (wm * WTM + (lane & 31)) * ROW_BYTES;
    const int qrow0 = (BM + wn * WTN + (lane & 31)) * ROW_BYTES;
    const int half = lane >> 5;

    Frags f0, f1;
    wait_stage(min(nk - 1, STAGES - 1));   // stages 1..3 may still be in flight
    raw_barrier();
    read_frags<NQ>(lds, prow0, qrow0, half, sw, f0);
    // Steady state (stage kt+4 exists): straight-line code with constant
    // waits, so the compiler's wait-count tracking sees that the fragments
    // multiplied were already waited for at the barrier and does not make
    // the multiplies wait for the reads of the next stage.
    auto steady = [&](int kt, Frags& cur, Frags& nxt) {
      wait_vmcnt<(STAGES - 2) * LOADS>();    // stage kt+1 landed, kt+2..kt+3 in flight
      __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): own reads of stage kt done
      raw_barrier();
      __builtin_amdgcn_sched_barrier(0);
      issue(prs, qrs, goff, (kt + STAGES) * BK, lds + (kt % STAGES) * STAGE_BYTES, w);
      read_frags<NQ>(lds + ((kt + 1) % STAGES) * STAGE_BYTES, prow0, qrow0, half, sw, nxt);
      mma<NQ>(cur, acc);
      interleave<NQ>();
      __builtin_amdgcn_sched_barrier(0);
    };
    // Last stages: fewer loads in flight, no more issues.
    auto step = [&](int kt, Frags& cur, Frags& nxt) {
      if (kt + 1 < nk) {
        // issued so far: stages up to min(nk-1, kt+3); stage kt+4 comes below
        wait_stage(min(nk - 1, kt + STAGES - 1) - (kt + 1));
        __builtin_amdgcn_s_waitcnt(0xC07F);
        raw_barrier();
        if (kt + STAGES < nk)
          issue(prs, qrs, goff, (kt + STAGES) * BK, lds + (kt % STAGES) * STAGE_BYTES, w);
        read_frags<NQ>(lds + ((kt + 1) % STAGES) * STAGE_BYTES, prow0, qrow0, half, sw, nxt);
      }
      mma<NQ>(cur, acc);
    };
    int kt = 0;
    for (; kt + 1 + STAGES < nk; kt += 2) {
      steady(kt, f0, f1);
      steady(kt + 1, f1, f0);
    }
    for (; kt + 1 < nk; kt += 2) {
      step(kt, f0, f1);
      step(kt + 1, f1, f0);
    }
    if (kt < nk) step(kt, f0, f1);
    __syncthreads();
  }

  // Same contract as run() with one fragment set: each stage's fragments are
  // read after its barrier and multiplied right away.  Fewer live registers,
  // for kernels whose epilogue needs them (the similarity tiles).
  static __device__ __forceinline__ void run_single(const uint16_t* __restrict__ pbase,
                                                    const uint32_t (&poff)[LOADS / 2],
                                                    const uint16_t* __restrict__ qbase,
                                                    const uint32_t (&qoff)[LOADS / 2], int K,
                                                    uint8_t* lds_generic, Acc& acc) {
    const lds_ptr lds = (lds_ptr)lds_generic;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = wave();
    const int wm = wave_m(w), wn = wave_n(w);
    const __amdgpu_buffer_rsrc_t prs = rsrc(pbase), qrs = rsrc(qbase);
    uint32_t goff[LOADS];
    dma_offsets(poff, qoff, goff);
    const int nk = K / BK;
#pragma unroll
    for (int st = 0; st < STAGES - 1; ++st)
      if (st < nk) issue(prs, qrs, goff, st * BK, lds + st * STAGE_BYTES, w);
    const int sw = swz(lane & 31);
    const int prow0 = (wm * WTM + (lane & 31)) * ROW_BYTES;
    const int qrow0 = (BM + wn * WTN + (lane & 31)) * ROW_BYTES;
    const int half = lane >> 5;
    for (int kt = 0; kt < nk; ++kt) {
      // issued: stages up to min(nk-1, kt+2)
      wait_stage(min(nk - 1, kt + STAGES - 2) - kt);
      raw_barrier();
      if (kt + STAGES - 1 < nk)
        issue(prs, qrs, goff, (kt + STAGES - 1) * BK, lds + ((kt + STAGES - 1) % STAGES) * STAGE_BYTES, w);
      Frags f;
      read_frags(lds + (kt % STAGES) * STAGE_BYTES, prow0, qrow0, half, sw, f);
      mma(f, acc);
    }
    __syncthreads();
  }
};

// Split-K for persistent kernels with fewer output tiles than CUs: each
// output tile's K range is cut into S parts that run as separate tiles and
// store float32 partial tiles; a separate reduction kernel (the kernel
// boundary makes the partials visible across XCDs) adds them in part order.
template <class G>
struct SplitK {
  static constexpr int MAX_SLOTS = 512;                       // >= CUs
  static constexpr size_t SLOT_FLOATS = static_cast<size_t>(G::BM) * G::BN;

  // parts per output tile: fill the grid once, at most 4, >= 4 K-stages each
  static __device__ __forceinline__ int parts(int tiles, int grid, int nk) {
    const int cap = min(grid, MAX_SLOTS);
    if (tiles <= 0 || tiles * 2 > cap) return 1;
    return max(1, min(min(cap / tiles, 4), nk / 4));
  }
};

// 512 threads, wave tile 128 x 64.
using GemmBig = Gemm256<2, 4>;
// 512 threads, wave tile 64 x 128; SIMD s holds P rows 64s..64s+63 of both
// Q halves (for Q tiles with a ragged number of valid rows).
using GemmRagged = Gemm256<4, 2, true>;
// 256 threads, wave tile 128 x 128 (accumulators fill the AGPRs).
using GemmWide = Gemm256<2, 2>;

// Persistent-kernel block order: consecutive virtual ids share an XCD
// (workgroups are dealt to the 8 XCDs round-robin), so the tiles that run
// together on one XCD are neighbours in tile order and share its L2.
__device__ __forceinline__ int xcd_virtual_block() {
  constexpr int kXcds = 8;
  const int g = gridDim.x, b = blockIdx.x;
  if (g % kXcds) return b;
  return (b % kXcds) * (g / kXcds) + b / kXcds;
}

}  // namespace luffy
