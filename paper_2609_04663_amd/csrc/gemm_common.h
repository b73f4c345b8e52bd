// Device helpers shared by the multi-product GEMM kernels.
#pragma once

#include "emu_internal.h"

#include <utility>

namespace emu {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void *lds_void_ptr;

// Workgroup -> output tile.  The hardware hands workgroup i to XCD i % 8; the
// remap gives each XCD a contiguous run of tile ids, and tile ids walk the
// output in groups of GROUP_M tile-rows so that the workgroups resident on one
// XCD at a time share A row-panels and B column-panels in that XCD's L2.
// Tile of virtual workgroup w out of nwg (a persistent workgroup w0 of a grid of
// G, G a multiple of 8, takes w = w0, w0 + G, ...: the same XCD throughout).
template <int GROUP_M>
__device__ inline void tile_coords_of(int w, int nwg, int nt_m, int nt_n, int &tm, int &tn) {
    const int per = nwg / 8, rem = nwg % 8, x = w % 8, j = w / 8;
    const int id = (x < rem) ? x * (per + 1) + j : rem * (per + 1) + (x - rem) * per + j;
    const int group = GROUP_M * nt_n;
    const int g = id / group, first = g * GROUP_M;
    const int gm = min(nt_m - first, GROUP_M);
    const int r = id - g * group;
    tm = first + r % gm;
    tn = r / gm;
}
template <int GROUP_M>
__device__ inline void tile_coords(int nt_m, int nt_n, int &tm, int &tn) {
    tile_coords_of<GROUP_M>(blockIdx.x, gridDim.x, nt_m, nt_n, tm, tn);
}

// One 1 KB direct global->LDS copy by a wave: lane l moves 16 bytes from
// src_wave + 16 l to lds_dst + 16 l (src_wave and lds_dst must be uniform over
// the wave).  The source base is pinned to scalar registers so that the copy
// takes the scalar-base form (64-bit base in SGPRs, 32-bit lane offset in one
// VGPR shared by every copy) instead of a 64-bit address per lane; that form
// holds the issuing wave for fewer cycles.
__device__ inline void copy_1k(const char *src_wave, char *lds_dst, unsigned lane16) {
    asm volatile("" : "+s"(src_wave));
    asm volatile("" : "+v"(lane16));   // keeps the offset 32-bit at the copy (no hoisted widening)
    __builtin_amdgcn_global_load_lds((const void *)(src_wave + lane16), (lds_void_ptr)lds_dst, 16,
                                     0, 0);
}

// Per-lane byte offset, inside a [rows][64 B] LDS tile, of the MFMA operand
// fragment of a 32-row block for reduction sub-step s (16 indices): lane l
// reads row (l % 32), 16-byte chunk q = 2 s + l / 32, swizzled as packed.
__device__ inline int frag_offset(int lane, int s) {
    const int row = lane & 31;
    const int q = 2 * s + (lane >> 5);
    return row * 64 + ((q ^ swz(row)) << 4);
}

__device__ inline bf16x8 lds_frag(const char *tile_block, int off) {
    return *reinterpret_cast<const bf16x8 *>(tile_block + off);
}

__device__ inline f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// MFMA whose accumulator is pinned to VGPRs (the builtin's accumulators live
// in AGPRs; a kernel with more than 256 accumulator registers would otherwise
// have them shuffled between the two files every iteration).  The compiler
// does not see inside the asm, so a VALU read of the result must go through
// mfma_vacc_settle first (wait states for the MFMA write, see below).
__device__ inline void mfma_vacc(f32x16 &c, bf16x8 a, bf16x8 b) {
    asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(c) : "v"(a), "v"(b));
}
__device__ inline void mfma_vacc_zero(f32x16 &c, bf16x8 a, bf16x8 b) {
    asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=v"(c) : "v"(a), "v"(b));
}
// Wait states before VALU instructions may read an inline-asm MFMA result
// (the hardware does not interlock this; 24 is above what a 32x32x16 MFMA
// needs).  Taking c as an operand orders every later reader after it.
__device__ inline void mfma_vacc_settle(f32x16 &c) {
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+v"(c));
}

// The same for the 16 x 16 x 32 MFMA (lane l holds A row l % 16 and B column
// l % 16 over reduction indices 8 (l / 16) .. 8 (l / 16) + 7; accumulator
// register r of lane l is output row 4 (l / 16) + r, column l % 16).
__device__ inline f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ inline void mfma16_vacc(f32x4 &c, bf16x8 a, bf16x8 b) {
    asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+v"(c) : "v"(a), "v"(b));
}
__device__ inline void mfma16_vacc_zero(f32x4 &c, bf16x8 a, bf16x8 b) {
    asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0" : "=v"(c) : "v"(a), "v"(b));
}
__device__ inline void mfma16_vacc_settle(f32x4 &c) {
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+v"(c));
}

// Workgroup barrier for the k-loop pipeline.  The caller has already issued
// the s_waitcnt it needs (its own LDS reads done, its copies of the next stage
// landed); unlike __syncthreads() this does not also wait for the copies that
// are still meant to be in flight.  The empty asm statements keep the compiler
// from moving memory accesses across the barrier.
__device__ inline void pipeline_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// f(std::integral_constant<int, I>) for I = 0 .. N - 1, in order, with I a
// constant expression inside f (for instruction sequences fixed at compile time).
template <typename F, int... I>
__device__ inline void static_for_impl(F &f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ inline void static_for(F &&f) {
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Scheduling fence that lets only VALU and SALU instructions (address
// arithmetic) move across it: MFMA, LDS and global memory instructions keep
// their program order.
__device__ inline void order_fence() { __builtin_amdgcn_sched_barrier(0x6); }

// Output update of the BLAS form C = alpha P + beta C, rounded as
// fl(fl(alpha P) + fl(beta C)) with no contraction; beta == 0 never reads C
// (BLAS convention: C may hold anything), and alpha == 1, beta == 0 stores P.
// (The operations are written here, under the pragma, rather than through
// helper functions whose inlined bodies would still be contracted.)
__device__ inline double out_update(double p, double alpha, double beta, const double *c) {
#pragma clang fp contract(off)
    const double ap = alpha * p;
    if (beta == 0.0) return ap;
    const double bc = beta * *c;
    return ap + bc;
}
__device__ inline float out_update(float p, float alpha, float beta, const float *c) {
#pragma clang fp contract(off)
    const float ap = alpha * p;
    if (beta == 0.0f) return ap;
    const float bc = beta * *c;
    return ap + bc;
}

// Output coordinates of accumulator register r of lane l in a 32x32 block:
// row (r / 4) * 8 + (l / 32) * 4 + r % 4, column l % 32.
__device__ inline int acc_row(int lane, int r) { return (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3); }

}  // namespace emu
