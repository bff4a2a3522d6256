// Inline-assembly building blocks of the pipelined bf16 map kernels (device
// code only): buffer loads into LDS, stores, LDS reads and writes with
// explicit wait counts, and matrix instructions that take their A operand
// from AGPRs.  Every memory instruction is issued from inline assembly so that
// it keeps its place in the stream; the kernels count them for their waits.
#pragma once

#include "kvx_bf16.h"

namespace kvx {
namespace {

typedef int i32x4_t __attribute__((ext_vector_type(4)));

// Buffer resource over [base, base + bytes): raw addressing, range-checked
// (reads outside return zero, writes outside are dropped).
__device__ __forceinline__ i32x4_t make_rsrc(const void* base, uint32_t bytes) {
  const uint64_t p = (uint64_t)(uintptr_t)base;
  i32x4_t r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)p);
  r[1] = __builtin_amdgcn_readfirstlane((int)((uint32_t)(p >> 32) & 0xffffu));
  r[2] = __builtin_amdgcn_readfirstlane((int)bytes);
  r[3] = 0x00020000;
  return r;
}

// 16 (or 4) bytes per lane from buffer r at voff into LDS at lds + 16 * lane
// (lds + 4 * lane), soffset 0.  The range check of a buffer covers voffset but
// not soffset, so loads that may reach past the end of a range carry their
// whole offset in voff.  The statement carries five wait states after any
// vector write of an SGPR it reads and the one after the write of M0; the
// _near forms only the latter (their operands were formed well before).
__device__ __forceinline__ void dma16z(uint32_t lds, uint32_t voff, const i32x4_t& r) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 4\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(r)
               : "memory");
}
__device__ __forceinline__ void dma16z_near(uint32_t lds, uint32_t voff, const i32x4_t& r) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(r)
               : "memory");
}
__device__ __forceinline__ void dma4z(uint32_t lds, uint32_t voff, const i32x4_t& r) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 4\n\tbuffer_load_dword %1, %2, 0 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(r)
               : "memory");
}
__device__ __forceinline__ void dma4z_near(uint32_t lds, uint32_t voff, const i32x4_t& r) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, 0 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(r)
               : "memory");
}

// 16 bytes per lane from buffer r at voff + soff into LDS at lds + 16 * lane.
// Inline assembly hides its operands from the compiler's hazard checks, so
// the statement carries its own wait states: five after any vector write of
// an SGPR it reads (the offset may come from v_readfirstlane), which also
// covers the one after the write of M0.
__device__ __forceinline__ void dma16(uint32_t lds, uint32_t voff, const i32x4_t& r, uint32_t soff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 4\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(r), "s"(soff)
               : "memory");
}

// The same load for operands produced well before it: soff and r must not
// have been written by a vector instruction (v_readfirstlane) within the
// five preceding wait states; only the wait state after the write of M0 is
// part of the statement.
__device__ __forceinline__ void dma16_near(uint32_t lds, uint32_t voff, const i32x4_t& r, uint32_t soff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(r), "s"(soff)
               : "memory");
}
__device__ __forceinline__ void dma4_near(uint32_t lds, uint32_t voff, const i32x4_t& r, uint32_t soff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, %3 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(r), "s"(soff)
               : "memory");
}

// 4 bytes per lane, the same way (lds + 4 * lane).
__device__ __forceinline__ void dma4(uint32_t lds, uint32_t voff, const i32x4_t& r, uint32_t soff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 4\n\tbuffer_load_dword %1, %2, %3 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(r), "s"(soff)
               : "memory");
}

// Stores through buffer r, from inline assembly so that every memory
// instruction keeps its place.  A store of more than 8 bytes reads its data
// registers after issue: the two wait states that the compiler would insert
// before the next write of those registers are part of the statement, and so
// are five before it (its buffer descriptor is read from SGPRs).
template <int OFF>
__device__ __forceinline__ void vstore16(const u32x4_t& v, uint32_t voff, const i32x4_t& r) {
  asm volatile("s_nop 4\n\tbuffer_store_dwordx4 %0, %1, %2, 0 offen offset:%3\n\ts_nop 1"
               :
               : "v"(v), "v"(voff), "s"(r), "n"(OFF)
               : "memory");
}

// The same store when r was written long before (see dma16_near).
template <int OFF>
__device__ __forceinline__ void vstore16_near(const u32x4_t& v, uint32_t voff, const i32x4_t& r) {
  asm volatile("buffer_store_dwordx4 %0, %1, %2, 0 offen offset:%3\n\ts_nop 1"
               :
               : "v"(v), "v"(voff), "s"(r), "n"(OFF)
               : "memory");
}

// Wait until at most N vector memory operations are outstanding.  Loads into
// LDS retire in order among themselves; they are not ordered with stores, so
// a wait for a load into LDS counts only the loads into LDS issued after it
// (outstanding stores only make the wait longer).
template <int N>
__device__ __forceinline__ void vm_wait() { asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory"); }

template <int OFF>
__device__ __forceinline__ void lds_read(u32x4_t& v, uint32_t addr) {
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "n"(OFF));
}
template <int OFF>
__device__ __forceinline__ void lds_write(uint32_t addr, const u32x4_t& v) {
  asm volatile("ds_write_b128 %0, %1 offset:%2" : : "v"(addr), "v"(v), "n"(OFF) : "memory");
}
template <int N>
__device__ __forceinline__ void lds_wait(u32x4_t& a) { asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(a) : "n"(N)); }
template <int N>
__device__ __forceinline__ void lds_wait2(u32x4_t& a, u32x4_t& b) {
  asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(a), "+v"(b) : "n"(N));
}
// Two 8-byte reads, at addr + 8 * O0 and addr + 8 * O1, into one register
// quadruple.
template <int O0, int O1>
__device__ __forceinline__ void lds_read2_b64(u32x4_t& v, uint32_t addr) {
  asm volatile("ds_read2_b64 %0, %1 offset0:%2 offset1:%3" : "=v"(v) : "v"(addr), "n"(O0), "n"(O1));
}
__device__ __forceinline__ void lds_read_b32(uint32_t& v, uint32_t addr) {
  asm volatile("ds_read_b32 %0, %1" : "=v"(v) : "v"(addr));
}
__device__ __forceinline__ void lds_wait_n(int n, u32x4_t& a) {
  switch (n) {
    case 0: lds_wait<0>(a); break;
    case 1: lds_wait<1>(a); break;
    case 2: lds_wait<2>(a); break;
    case 3: lds_wait<3>(a); break;
    case 4: lds_wait<4>(a); break;
    case 5: lds_wait<5>(a); break;
    case 6: lds_wait<6>(a); break;
    case 7: lds_wait<7>(a); break;
    case 8: lds_wait<8>(a); break;
    case 9: lds_wait<9>(a); break;
    case 10: lds_wait<10>(a); break;
    case 11: lds_wait<11>(a); break;
    case 12: lds_wait<12>(a); break;
    case 13: lds_wait<13>(a); break;
    case 14: lds_wait<14>(a); break;
    default: lds_wait<15>(a); break;
  }
}
__device__ __forceinline__ void lds_drain() { asm volatile("s_waitcnt lgkmcnt(0)" : : : "memory"); }

__device__ __forceinline__ uint32_t lds_u32(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// acc = A * B + acc, and acc = A * B + C with A (the map) in AGPRs.
__device__ __forceinline__ void mfma_acc(f32x4_t& acc, const u32x4_t& w, const u32x4_t& x) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+v"(acc) : "a"(w), "v"(x));
}
__device__ __forceinline__ void mfma_zero(f32x4_t& acc, const u32x4_t& w, const u32x4_t& x) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0" : "=&v"(acc) : "a"(w), "v"(x));
}
__device__ __forceinline__ void mfma_init(f32x4_t& acc, const u32x4_t& w, const u32x4_t& x,
                                          const f32x4_t& c) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %3" : "=&v"(acc) : "a"(w), "v"(x), "v"(c));
}

// Pin values to a point of the instruction stream (between two matrix
// instructions): they are produced before it and consumed after it.
template <typename A>
__device__ __forceinline__ void pin(A& a) { asm volatile("" : "+v"(a)); }
template <typename A, typename B>
__device__ __forceinline__ void pin(A& a, B& b) { asm volatile("" : "+v"(a), "+v"(b)); }
template <typename A, typename B, typename C, typename E>
__device__ __forceinline__ void pin(A& a, B& b, C& c, E& e) {
  asm volatile("" : "+v"(a), "+v"(b), "+v"(c), "+v"(e));
}

}  // namespace
}  // namespace kvx
