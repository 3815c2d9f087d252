// LDS DMA helpers shared by the bf16 expert GEMMs: global -> LDS copies with
// global_load_lds_dwordx4 (no VGPR staging) and exact vmcnt waits.
//
// An "8-row unit" is what one DMA instruction moves: 8 rows x 128 bytes (a
// 64-wide bf16 K stage of 8 rows, whole cache lines).  DMA lane i lands at
// byte 16*i, i.e. row i/8, slot i%8; the lane fetches chunk (i%8) ^ (i/8) of
// its row, so chunk c of row r sits in slot c ^ r.  A 16-row block is two
// consecutive units with the same permutation; lane l's operand of
// v_mfma_f32_16x16x32_bf16 (row l%16, 8 k values 32h + 8(l/16) .. +7 of k half
// h) is read from unit_read_offset(l, h).  Measured on gfx950 (ds_read_b128,
// 8 waves per CU): this read pattern runs at the full LDS rate (~236 bytes per
// clock per CU, as for 16 lanes reading one contiguous 256-byte block) at any
// 1 KB-aligned block base; giving the second unit another permutation (slot c ^
// r ^ 1, which is bank-distinct under a plain address-modulo bank map) halves
// it, so the bank map evidently folds in address bits above the 256-byte row.
#pragma once

#include "ace_internal.h"

namespace ace {

constexpr int kUnitBytes = 1024;  // one 8-row unit (and one 16 x 32 MFMA fragment)

__device__ __forceinline__ uint32_t lds_addr(const void *p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const void *)p));
}

// chunk (16 bytes, 8 bf16) of its row that DMA lane `lane` fetches (either unit
// of a 16-row block)
__host__ __device__ inline int unit_chunk(int lane) { return (lane & 7) ^ (lane >> 3); }

// byte offset, from a 16-row block's first unit, of lane's MFMA operand for k half h
__host__ __device__ inline int unit_read_offset(int lane, int h) {
  const int r16 = lane & 15, g = lane >> 4, rlo = r16 & 7, uh = r16 >> 3;
  return uh * kUnitBytes + rlo * 128 + (((4 * h + g) ^ rlo) << 4);
}

// 16 bytes per lane from global `src` into LDS at lds_base + 16 * lane.  M0 is
// declared clobbered, so the compiler sets it again wherever it needs it (saving
// and restoring it around every DMA cost the matrix-bound tiles about 1%).
// An SALU write of M0 needs one wait state before a global load with the LDS bit
// reads it (the ISA's table of manually inserted wait states; the compiler's
// hazard check does not see inside this asm), hence the s_nop.
// The compiler does not see this LDS write: every consumer waits on vmcnt
// explicitly (and crosses a barrier when another wave issued the copy).
__device__ __forceinline__ void dma16(const void *src, uint32_t lds_base) {
  asm volatile(
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, off"
      :
      : "v"(src), "s"(__builtin_amdgcn_readfirstlane(lds_base))
      : "memory", "m0");
}

// dma16 with the non-temporal cache hint (nt), for data each launch reads once:
// the expert weights.  Streaming them this way leaves the caches to the layer's
// reused data (activation rows, H and Y between kernels, the router rows); the
// decode GEMMs stream about 10% faster with it.
__device__ __forceinline__ void dma16_stream(const void *src, uint32_t lds_base) {
  asm volatile(
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, off nt"
      :
      : "v"(src), "s"(__builtin_amdgcn_readfirstlane(lds_base))
      : "memory", "m0");
}

__device__ __forceinline__ void barrier() { asm volatile("s_barrier" ::: "memory"); }

// A 32-bit load the compiler does not track: it places no wait for it.  The
// caller waits with wait_vmcnt (counting this load in its issue order) and then
// passes the value through reg_ready before reading it.
__device__ __forceinline__ int gload_i32(const int32_t *p) {
  int v;
  asm volatile("global_load_dword %0, %1, off" : "=v"(v) : "v"(p) : "memory");
  return v;
}
__device__ __forceinline__ void reg_ready(int &v) { asm volatile("" : "+v"(v)::"memory"); }

// wait until at most n (0..63) of this wave's vector memory operations are outstanding
__device__ __forceinline__ void wait_vmcnt(int n) {
#define ACE_VMCNT_CASE(c) \
  case c:                 \
    asm volatile("s_waitcnt vmcnt(" #c ")" ::: "memory"); \
    break;
  switch (n) {
    ACE_VMCNT_CASE(0) ACE_VMCNT_CASE(1) ACE_VMCNT_CASE(2) ACE_VMCNT_CASE(3) ACE_VMCNT_CASE(4)
    ACE_VMCNT_CASE(5) ACE_VMCNT_CASE(6) ACE_VMCNT_CASE(7) ACE_VMCNT_CASE(8) ACE_VMCNT_CASE(9)
    ACE_VMCNT_CASE(10) ACE_VMCNT_CASE(11) ACE_VMCNT_CASE(12) ACE_VMCNT_CASE(13) ACE_VMCNT_CASE(14)
    ACE_VMCNT_CASE(15) ACE_VMCNT_CASE(16) ACE_VMCNT_CASE(17) ACE_VMCNT_CASE(18) ACE_VMCNT_CASE(19)
    ACE_VMCNT_CASE(20) ACE_VMCNT_CASE(21) ACE_VMCNT_CASE(22) ACE_VMCNT_CASE(23) ACE_VMCNT_CASE(24)
    ACE_VMCNT_CASE(25) ACE_VMCNT_CASE(26) ACE_VMCNT_CASE(27) ACE_VMCNT_CASE(28) ACE_VMCNT_CASE(29)
    ACE_VMCNT_CASE(30) ACE_VMCNT_CASE(31) ACE_VMCNT_CASE(32) ACE_VMCNT_CASE(33) ACE_VMCNT_CASE(34)
    ACE_VMCNT_CASE(35) ACE_VMCNT_CASE(36) ACE_VMCNT_CASE(37) ACE_VMCNT_CASE(38) ACE_VMCNT_CASE(39)
    ACE_VMCNT_CASE(40) ACE_VMCNT_CASE(41) ACE_VMCNT_CASE(42) ACE_VMCNT_CASE(43) ACE_VMCNT_CASE(44)
    ACE_VMCNT_CASE(45) ACE_VMCNT_CASE(46) ACE_VMCNT_CASE(47) ACE_VMCNT_CASE(48) ACE_VMCNT_CASE(49)
    ACE_VMCNT_CASE(50) ACE_VMCNT_CASE(51) ACE_VMCNT_CASE(52) ACE_VMCNT_CASE(53) ACE_VMCNT_CASE(54)
    ACE_VMCNT_CASE(55) ACE_VMCNT_CASE(56) ACE_VMCNT_CASE(57) ACE_VMCNT_CASE(58) ACE_VMCNT_CASE(59)
    ACE_VMCNT_CASE(60) ACE_VMCNT_CASE(61) ACE_VMCNT_CASE(62) ACE_VMCNT_CASE(63)
    default: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
  }
#undef ACE_VMCNT_CASE
}

}  // namespace ace
