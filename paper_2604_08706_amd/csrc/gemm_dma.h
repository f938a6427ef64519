// bf16 MFMA mainloop for two K-major operands with HBM -> LDS direct loads
// (gfx950 buffer_load_dwordx4 ... lds), used where both operands are stored
// with k contiguous.  Same workgroup tile, wave grid, MFMA and accumulator
// layout as gemm_core.h, so the epilogues work on either mainloop.
//
// K step 32, four LDS stages of 32 KiB (A then B, each [256 rows][32 k] bf16 =
// 64-byte rows).  The loads of step s + 3 are issued two iterations before
// step s + 3 is multiplied, straight into LDS: no staging registers, no
// ds_write instructions, and ~2000 MFMA cycles of latency cover.
//
// The loads are issued with inline assembly and their completion is tracked by
// hand (s_waitcnt vmcnt): the compiler's own tracking of LDS-DMA would wait for
// every outstanding load before each LDS read and serialize the pipeline.
// Nothing else in these kernels touches M0 or issues vector memory loads inside
// the loop, and the loop ends with vmcnt(0).
//
// A DMA instruction writes 64 lanes x 16 bytes to LDS at M0 + 16 * lane, i.e.
// 16 consecutive 64-byte rows.  The bank swizzle is applied on the HBM side:
// the lane that lands on physical chunk p of row `row` fetches logical chunk
// p ^ f(row) with f(row) = ((row >> 1) ^ (row >> 2)) & 3, which makes every
// fragment read (32 consecutive rows, one chunk) hit distinct banks whether the
// LDS serves 8 or 16 lanes of a 16-byte read per cycle.
#pragma once

#include "gemm_core.h"

namespace rbp {
namespace gemm {

constexpr int kDmaBK = 32;
constexpr int kDmaStages = 4;
constexpr int kDmaTile = 256 * kDmaBK * 2;   // 16 KiB
constexpr int kDmaStage = 2 * kDmaTile;      // A + B
constexpr int kDmaLds = kDmaStages * kDmaStage;
static_assert(kDmaLds <= kLdsBytes, "DMA stages must fit the shared LDS allocation");

typedef int i32x4 __attribute__((ext_vector_type(4)));

// Raw buffer resource as four SGPRs: 48-bit base, stride 0, range in bytes.
__device__ __forceinline__ i32x4 rsrc_words(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  return i32x4{(int)(uint32_t)a, (int)((a >> 32) & 0xffffu), (int)bytes, 0x00020000};
}

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// 16 bytes per lane from buffer offset `voff` into LDS at lds + 16 * lane.
__device__ __forceinline__ void dma16(uint32_t lds, uint32_t voff, i32x4 rsrc) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(rsrc)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// s_waitcnt encodings (gfx9): vmcnt in bits [3:0] and [15:14], expcnt [6:4],
// lgkmcnt [11:8]; other counters left at their maximum.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xf << 8));
}

// Workgroup barrier that is also a compiler memory barrier: LDS reads after it
// may not be moved above it (s_barrier alone orders no memory accesses).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Wave grid of a DMA workgroup: WM x WN waves over the 256 x 256 tile, each
// wave owning (256 / WM) x (256 / WN) outputs = MI x NI MFMA tiles of 32 x 32.
template <int WM_, int WN_>
struct Grid {
  static constexpr int WM = WM_, WN = WN_;
  static constexpr int kWaves = WM * WN;
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int MI = 256 / 32 / WM;
  static constexpr int NI = 256 / 32 / WN;
  static constexpr int kLoadsPerOperand = 16 / kWaves;  // 1 KiB blocks per wave per step
  static __device__ __forceinline__ int wave() { return threadIdx.x >> 6; }
  static __device__ __forceinline__ int wm() { return wave() / WN; }
  static __device__ __forceinline__ int wn() { return wave() % WN; }
  // row (m) / column (n) of accumulator r of MFMA tile (mi, ni), tile-relative
  static __device__ __forceinline__ int row(int mi, int r) {
    return wm() * (256 / WM) + mi * 32 + (r >> 2) * 8 + ((threadIdx.x & 63) >> 5) * 4 + (r & 3);
  }
  static __device__ __forceinline__ int col(int ni) {
    return wn() * (256 / WN) + ni * 32 + (threadIdx.x & 31);
  }
};
using Grid4 = Grid<2, 2>;  // 4 waves, 128 x 128 per wave
using Grid8 = Grid<2, 4>;  // 8 waves (two per SIMD), 128 x 64 per wave

// Per-thread load plan of one K-major operand tile (256 rows x 32 k).
template <class G>
struct DmaOperand {
  i32x4 rsrc;
  uint32_t voff0;      // byte offset of this lane's chunk for j = 0 at k = 0
  uint32_t row_step;   // bytes between the row blocks of j and j + 1
  int kc;              // first k of this lane's chunk within the step
  int64_t k_extent;

  __device__ __forceinline__ void init(const Operand& op, int64_t mn0) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int64_t rows = op.mn_extent - mn0;
    rows = rows < 0 ? 0 : (rows > 256 ? 256 : rows);
    rsrc = rsrc_words(op.ptr + mn0 * op.ld, (uint32_t)(rows * op.ld * 2));
    // block j * kWaves + wave holds 16 rows; lane -> row + lane/4, physical
    // chunk lane % 4, logical chunk (lane % 4) ^ f(row), f(row) the same for
    // every block because blocks start at multiples of 16 rows
    const int row = wave * 16 + (lane >> 2);
    const int f = ((lane >> 3) ^ (lane >> 4)) & 3;
    const int c = (lane & 3) ^ f;
    kc = c * 8;
    voff0 = (uint32_t)((row * op.ld + kc) * 2);
    row_step = (uint32_t)(G::kWaves * 16 * op.ld * 2);
    k_extent = op.k_extent;
  }
  // Issue load j of this wave's loads of one step into the tile at LDS byte
  // address `tile` (step K offset k0).
  __device__ __forceinline__ void issue_one(uint32_t tile, int64_t k0, int j) const {
    const uint32_t wave = (uint32_t)__builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const bool ok = k0 + kc < k_extent;
    dma16(tile + (uint32_t)(j * G::kWaves + wave) * 1024u,
          ok ? voff0 + j * row_step + (uint32_t)(k0 * 2) : kOutOfRange, rsrc);
  }
  __device__ __forceinline__ void issue(uint32_t tile, int64_t k0) const {
#pragma unroll
    for (int j = 0; j < G::kLoadsPerOperand; ++j) issue_one(tile, k0, j);
  }
};

// Per-lane fragment bases for 64-byte rows: slice ks reads physical chunk
// (2 ks) ^ t with t = (lane / 32) ^ f(lane % 32) (fragment row blocks start at
// multiples of 32 rows, which leave f unchanged).
struct DmaFrag {
  uint32_t a[2], b[2];
};

template <class G>
__device__ __forceinline__ DmaFrag dma_frag_bases() {
  const int lane = threadIdx.x & 63;
  const int r = lane & 31;
  const int t = (lane >> 5) ^ (((r >> 1) ^ (r >> 2)) & 3);
  DmaFrag f;
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    const uint32_t off = (uint32_t)(r * 64 + (((2 * ks) ^ t) << 4));
    f.a[ks] = (uint32_t)(G::wm() * (256 / G::WM) * 64) + off;
    f.b[ks] = (uint32_t)(kDmaTile + G::wn() * (256 / G::WN) * 64) + off;
  }
  return f;
}

template <class G>
__device__ __forceinline__ void dma_frags(const uint8_t* stage, const DmaFrag& f, int ks,
                                          bf16x8 (&a)[G::MI], bf16x8 (&b)[G::NI]) {
#pragma unroll
  for (int i = 0; i < G::MI; ++i)
    a[i] = *reinterpret_cast<const bf16x8*>(stage + f.a[ks] + 2048 * i);
#pragma unroll
  for (int i = 0; i < G::NI; ++i)
    b[i] = *reinterpret_cast<const bf16x8*>(stage + f.b[ks] + 2048 * i);
}

template <class G>
__device__ __forceinline__ void mfma_tiles(const bf16x8 (&a)[G::MI], const bf16x8 (&b)[G::NI],
                                           f32x16 (&acc)[G::MI][G::NI]) {
#pragma unroll
  for (int mi = 0; mi < G::MI; ++mi)
#pragma unroll
    for (int ni = 0; ni < G::NI; ++ni)
      acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mi], b[ni], acc[mi][ni], 0, 0, 0);
}

// MFMAs of one K slice with `nload` loads spread evenly between them: a
// burst of loads would stall this wave's MFMA issue while the CU's address
// unit accepts them.  load(l) issues load l (or nothing).
template <class G, class LoadFn>
__device__ __forceinline__ void mfma_tiles_interleaved(const bf16x8 (&a)[G::MI],
                                                       const bf16x8 (&b)[G::NI],
                                                       f32x16 (&acc)[G::MI][G::NI], int nload,
                                                       LoadFn&& load) {
  constexpr int M = G::MI * G::NI;
  const int every = M / nload;
#pragma unroll
  for (int q = 0; q < M; ++q) {
    const int mi = q / G::NI, ni = q % G::NI;
    acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mi], b[ni], acc[mi][ni], 0, 0, 0);
    if ((q + 1) % every == 0 && (q + 1) / every <= nload) {
      RBP_FENCE();
      load((q + 1) / every - 1);
      RBP_FENCE();
    }
  }
}

// vmcnt wait allowing `steps` later K steps (`per` loads each) to stay in flight.
template <int per>
__device__ __forceinline__ void wait_steps(int steps) {
  static_assert(kDmaStages <= 5, "extend the cases below");
  switch (steps) {
    case 0: wait_vmcnt<0>(); break;
    case 1: wait_vmcnt<per>(); break;
    case 2: wait_vmcnt<2 * per>(); break;
    default: wait_vmcnt<3 * per>(); break;
  }
}

// Full K loop over [k_begin, k_end) for the tile at (m0, n0), both operands
// K-major (k_extent % 8 == 0).  Step s lives in stage s % kDmaStages.  Per
// iteration s:
//   read slice 1 fragments; MFMAs of slice 0;
//   wait for step s + 1's loads, barrier (step s + 1 now visible, stage of
//   step s - 1 free); issue step s + kDmaStages - 1 into that stage;
//   read step s + 1's slice 0 fragments; MFMAs of slice 1.
// Ends with a barrier, so the caller may reuse `smem` right away.
template <class G>
__device__ __forceinline__ void mainloop_dma(const Operand& A, const Operand& B, int64_t m0,
                                             int64_t n0, int64_t k_begin, int64_t k_end,
                                             uint8_t* smem, f32x16 (&acc)[G::MI][G::NI]) {
#pragma unroll
  for (int mi = 0; mi < G::MI; ++mi)
#pragma unroll
    for (int ni = 0; ni < G::NI; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mi][ni][r] = 0.0f;
  const int64_t nk = (k_end - k_begin + kDmaBK - 1) / kDmaBK;
  if (nk <= 0) return;
  constexpr int kPer = 2 * G::kLoadsPerOperand;  // loads per thread per step
  DmaOperand<G> la, lb;
  la.init(A, m0);
  lb.init(B, n0);
  const DmaFrag f = dma_frag_bases<G>();
  const uint32_t lds0 = (uint32_t)reinterpret_cast<uintptr_t>(smem);
  auto issue = [&](int64_t step, int stage) {
    const uint32_t st = lds0 + (uint32_t)stage * kDmaStage;
    la.issue(st, k_begin + step * kDmaBK);
    lb.issue(st + kDmaTile, k_begin + step * kDmaBK);
  };
  // prologue: steps 0 .. kDmaStages - 2 in flight, wait for step 0
  const int64_t pre = nk < kDmaStages - 1 ? nk : kDmaStages - 1;
#pragma unroll
  for (int s = 0; s < kDmaStages - 1; ++s)
    if (s < pre) issue(s, s);
  wait_steps<kPer>((int)pre - 1);
  lds_barrier();
  bf16x8 a0[G::MI], b0[G::NI], a1[G::MI], b1[G::NI];
  dma_frags<G>(smem, f, 0, a0, b0);
  int cur = 0;                     // stage of step it
  int ahead = kDmaStages - 1;      // stage of step it + kDmaStages - 1
  for (int64_t it = 0; it < nk; ++it) {
    const int nxt = cur + 1 == kDmaStages ? 0 : cur + 1;
    dma_frags<G>(smem + cur * kDmaStage, f, 1, a1, b1);
    RBP_FENCE();
    mfma_tiles<G>(a0, b0, acc);
    RBP_FENCE();
    // steps issued so far: 0 .. min(nk, it + kDmaStages - 1) - 1; step it + 1 must be in
    const int64_t issued = nk < it + kDmaStages - 1 ? nk : it + kDmaStages - 1;
    const int64_t later = issued - (it + 2);
    wait_steps<kPer>(later < 0 ? 0 : (int)later);
    lds_barrier();
    // unconditional (the last iteration re-reads a stale stage): a read under
    // a branch would make the compiler wait for it before the MFMAs below
    dma_frags<G>(smem + nxt * kDmaStage, f, 0, a0, b0);
    RBP_FENCE();
    // step it + kDmaStages - 1 goes into the stage of step it - 1, now free;
    // its loads are spread over this slice's MFMAs
    const bool more = it + kDmaStages - 1 < nk;
    const uint32_t st = lds0 + (uint32_t)ahead * kDmaStage;
    const int64_t kn = k_begin + (it + kDmaStages - 1) * kDmaBK;
    mfma_tiles_interleaved<G>(a1, b1, acc, kPer, [&](int l) {
      if (more) {
        if (l < G::kLoadsPerOperand)
          la.issue_one(st, kn, l);
        else
          lb.issue_one(st + kDmaTile, kn, l - G::kLoadsPerOperand);
      }
    });
    RBP_FENCE();
    cur = nxt;
    ahead = ahead + 1 == kDmaStages ? 0 : ahead + 1;
  }
  wait_vmcnt<0>();
  __syncthreads();
}

}  // namespace gemm
}  // namespace rbp
