// LDS helpers shared by the MFMA kernels: asynchronous global -> LDS loads
// (global_load_lds_dwordx4), barriers that leave those loads in flight, and
// fragment reads as inline asm.
//
// The compiler cannot tell an LDS read from the in-flight LDS-DMA loads it
// might alias, and waits for every pending vector-memory operation before a
// builtin LDS read.  The fragment reads are therefore inline asm; each asm
// block issues up to 8 reads and ends with s_waitcnt lgkmcnt(0), so its
// outputs are complete when the block ends and the compiler may copy, spill
// or reuse them freely.  Read latency still overlaps the MFMAs issued before
// the block.  The build checks the assembly for any use of an asm read's
// result before its wait.
#pragma once

#include "common.h"

namespace lmoe {

static __device__ __attribute__((aligned(16))) uint32_t g_zero16[4];  // zero-initialised, never written

typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ void dma16(const void* src, uint16_t* lds_wave_base) {
  __builtin_amdgcn_global_load_lds(src, (lds_void*)lds_wave_base, 16, 0, 0);
}

__device__ __forceinline__ void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }

// Reads per asm block (the LGKM counter never holds more than this many).
constexpr int kReadChunk = 8;
__device__ __forceinline__ uint32_t lds_addr(const uint16_t* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint16_t*)p;
}

template <int N> struct Rd128;
template <> struct Rd128<8> {
  __device__ static void run(u32x4* o, const uint32_t* a) {
    asm volatile("ds_read_b128 %0, %8\n ds_read_b128 %1, %9\n ds_read_b128 %2, %10\n ds_read_b128 %3, %11\n"
                 "ds_read_b128 %4, %12\n ds_read_b128 %5, %13\n ds_read_b128 %6, %14\n ds_read_b128 %7, %15\n"
                 "s_waitcnt lgkmcnt(0)"
                 : "=&v"(o[0]), "=&v"(o[1]), "=&v"(o[2]), "=&v"(o[3]), "=&v"(o[4]), "=&v"(o[5]), "=&v"(o[6]), "=&v"(o[7])
                 : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]), "v"(a[6]), "v"(a[7])
                 : "memory");
  }
};
template <> struct Rd128<4> {
  __device__ static void run(u32x4* o, const uint32_t* a) {
    asm volatile("ds_read_b128 %0, %4\n ds_read_b128 %1, %5\n ds_read_b128 %2, %6\n ds_read_b128 %3, %7\n"
                 "s_waitcnt lgkmcnt(0)"
                 : "=&v"(o[0]), "=&v"(o[1]), "=&v"(o[2]), "=&v"(o[3])
                 : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3])
                 : "memory");
  }
};
template <int N> struct RdTr;
template <> struct RdTr<8> {
  __device__ static void run(u32x2* o, const uint32_t* a) {
    asm volatile("ds_read_b64_tr_b16 %0, %8\n ds_read_b64_tr_b16 %1, %9\n ds_read_b64_tr_b16 %2, %10\n"
                 "ds_read_b64_tr_b16 %3, %11\n ds_read_b64_tr_b16 %4, %12\n ds_read_b64_tr_b16 %5, %13\n"
                 "ds_read_b64_tr_b16 %6, %14\n ds_read_b64_tr_b16 %7, %15\n"
                 "s_waitcnt lgkmcnt(0)"
                 : "=&v"(o[0]), "=&v"(o[1]), "=&v"(o[2]), "=&v"(o[3]), "=&v"(o[4]), "=&v"(o[5]), "=&v"(o[6]), "=&v"(o[7])
                 : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]), "v"(a[6]), "v"(a[7])
                 : "memory");
  }
};

// Split reads: the *Issue blocks start up to 8 reads and return at once; the
// outputs are pending until a following lds_wait(...) names them.  In between,
// the caller may only issue independent work (the MFMAs of the previous
// fragments); the build's ISA check rejects any compiled use of a pending
// register before the wait.
template <int N> struct Rd128Issue;
template <> struct Rd128Issue<4> {
  __device__ static void run(u32x4* o, const uint32_t* a) {
    asm volatile("ds_read_b128 %0, %4\n ds_read_b128 %1, %5\n ds_read_b128 %2, %6\n ds_read_b128 %3, %7"
                 : "=&v"(o[0]), "=&v"(o[1]), "=&v"(o[2]), "=&v"(o[3])
                 : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3])
                 : "memory");
  }
};
template <> struct Rd128Issue<8> {
  __device__ static void run(u32x4* o, const uint32_t* a) {
    asm volatile("ds_read_b128 %0, %8\n ds_read_b128 %1, %9\n ds_read_b128 %2, %10\n ds_read_b128 %3, %11\n"
                 "ds_read_b128 %4, %12\n ds_read_b128 %5, %13\n ds_read_b128 %6, %14\n ds_read_b128 %7, %15"
                 : "=&v"(o[0]), "=&v"(o[1]), "=&v"(o[2]), "=&v"(o[3]), "=&v"(o[4]), "=&v"(o[5]), "=&v"(o[6]), "=&v"(o[7])
                 : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]), "v"(a[6]), "v"(a[7])
                 : "memory");
  }
};
struct RdTrIssue8 {
  __device__ static void run(u32x2* o, const uint32_t* a) {
    asm volatile("ds_read_b64_tr_b16 %0, %8\n ds_read_b64_tr_b16 %1, %9\n ds_read_b64_tr_b16 %2, %10\n"
                 "ds_read_b64_tr_b16 %3, %11\n ds_read_b64_tr_b16 %4, %12\n ds_read_b64_tr_b16 %5, %13\n"
                 "ds_read_b64_tr_b16 %6, %14\n ds_read_b64_tr_b16 %7, %15"
                 : "=&v"(o[0]), "=&v"(o[1]), "=&v"(o[2]), "=&v"(o[3]), "=&v"(o[4]), "=&v"(o[5]), "=&v"(o[6]), "=&v"(o[7])
                 : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]), "v"(a[6]), "v"(a[7])
                 : "memory");
  }
};
__device__ __forceinline__ void lds_wait(u32x4 (&o)[4]) {
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(o[0]), "+v"(o[1]), "+v"(o[2]), "+v"(o[3]) :: "memory");
}
__device__ __forceinline__ void lds_wait(u32x4 (&o)[8]) {
  asm volatile("s_waitcnt lgkmcnt(0)"
               : "+v"(o[0]), "+v"(o[1]), "+v"(o[2]), "+v"(o[3]), "+v"(o[4]), "+v"(o[5]), "+v"(o[6]), "+v"(o[7])
               :: "memory");
}
__device__ __forceinline__ void lds_wait(u32x2 (&o)[8]) {
  asm volatile("s_waitcnt lgkmcnt(0)"
               : "+v"(o[0]), "+v"(o[1]), "+v"(o[2]), "+v"(o[3]), "+v"(o[4]), "+v"(o[5]), "+v"(o[6]), "+v"(o[7])
               :: "memory");
}
// Marks registers of reads that an earlier lds_wait in the same sequence has
// already retired (no instruction; keeps the compiler from touching them early).
__device__ __forceinline__ void lds_retired(u32x2 (&o)[8]) {
  asm volatile(""
               : "+v"(o[0]), "+v"(o[1]), "+v"(o[2]), "+v"(o[3]), "+v"(o[4]), "+v"(o[5]), "+v"(o[6]), "+v"(o[7])
               :: "memory");
}

// Single fragment reads for hand-interleaved schedules: the output is pending
// until a later s_waitcnt lgkmcnt(0) followed by lds_mark on it.
__device__ __forceinline__ void rd128_issue(u32x4& o, uint32_t a) {
  asm volatile("ds_read_b128 %0, %1" : "=v"(o) : "v"(a) : "memory");
}
__device__ __forceinline__ void rdtr_issue(u32x2& o, uint32_t a) {
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(o) : "v"(a) : "memory");
}
// The same with a constant byte offset in the instruction (0 .. 65535).
template <int OFF>
__device__ __forceinline__ void rd128_issue_at(u32x4& o, uint32_t a) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(o) : "v"(a), "n"(OFF) : "memory");
}
template <int OFF>
__device__ __forceinline__ void rdtr_issue_at(u32x2& o, uint32_t a) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(o) : "v"(a), "n"(OFF) : "memory");
}
__device__ __forceinline__ void lds_wait_all() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
// At most n LDS operations outstanding (keeps the 4-bit counter from overflowing).
template <int N>
__device__ __forceinline__ void lds_wait_le() {
  static_assert(N >= 0 && N < 16, "lgkmcnt range");
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
}
// Marks registers of reads retired by an earlier lds_wait_all (no instruction).
template <int N>
__device__ __forceinline__ void lds_mark(u32x4 (&o)[N]) {
#pragma unroll
  for (int i = 0; i < N; i += 4)
    asm volatile("" : "+v"(o[i]), "+v"(o[i + 1]), "+v"(o[i + 2]), "+v"(o[i + 3])::"memory");
}
template <int N>
__device__ __forceinline__ void lds_mark(u32x2 (&o)[N]) {
#pragma unroll
  for (int i = 0; i < N; i += 8)
    asm volatile(""
                 : "+v"(o[i]), "+v"(o[i + 1]), "+v"(o[i + 2]), "+v"(o[i + 3]), "+v"(o[i + 4]), "+v"(o[i + 5]),
                   "+v"(o[i + 6]), "+v"(o[i + 7])::"memory");
}

// vmcnt(n) (gfx9 encoding; expcnt and lgkmcnt unrestricted).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Wait until at most n * LPS vector-memory operations are pending (n <= NMAX, decided at run time).
template <int LPS, int NMAX>
__device__ __forceinline__ void wait_vm_tiles(int n) {
  if constexpr (NMAX <= 0) {
    wait_vm<0>();
  } else {
    if (n >= NMAX) wait_vm<NMAX * LPS>();
    else wait_vm_tiles<LPS, NMAX - 1>(n);
  }
}

}  // namespace lmoe
