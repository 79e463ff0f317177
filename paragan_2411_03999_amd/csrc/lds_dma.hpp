// Direct global-to-LDS loads and the waits of an LDS ring (gfx950).
#pragma once
#include "common.hpp"

namespace pg {

// Byte address in LDS of a pointer into a __shared__ array, made
// wave-uniform (it becomes the M0 base of a direct load).
PG_DEV uint32_t lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)(p));
}

// 16 bytes per lane from a buffer straight into LDS at M0 + 16 * lane (an
// out-of-range offset writes zeros).  Issued as inline assembly so that the
// compiler's wait-count insertion does not treat the stores into the other
// stages of the ring as hazards for every LDS read; their completion is
// waited for explicitly (wait_barrier), which is correct because the main
// loop issues no other vector-memory instructions.
// The byte address is voff (per lane) + soff (uniform).
PG_DEV void lds_load16(uint32_t lds_base, uint32_t voff, uint32_t soff, __amdgpu_buffer_rsrc_t r) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds" ::"s"(lds_base), "v"(voff),
               "s"(r), "s"(soff)
               : "memory", "m0");
}

// Wait until at most N of this wave's vector-memory loads are outstanding
// and all of its LDS reads have completed, then barrier: one statement, so
// nothing the compiler schedules can slip between the wait and the barrier.
template <int N>
PG_DEV void wait_barrier();
#define PG_WAIT_BARRIER(N)                                                          \
  template <>                                                                       \
  PG_DEV void wait_barrier<N>() {                                                   \
    asm volatile("s_waitcnt vmcnt(" #N ") lgkmcnt(0)\n\ts_barrier" ::: "memory");   \
  }
PG_WAIT_BARRIER(0)
PG_WAIT_BARRIER(1)
PG_WAIT_BARRIER(2)
PG_WAIT_BARRIER(3)
PG_WAIT_BARRIER(4)
PG_WAIT_BARRIER(5)
PG_WAIT_BARRIER(6)
PG_WAIT_BARRIER(7)
PG_WAIT_BARRIER(8)
PG_WAIT_BARRIER(9)
PG_WAIT_BARRIER(10)
PG_WAIT_BARRIER(11)
PG_WAIT_BARRIER(12)
PG_WAIT_BARRIER(13)
PG_WAIT_BARRIER(14)
PG_WAIT_BARRIER(15)
PG_WAIT_BARRIER(16)
PG_WAIT_BARRIER(17)
PG_WAIT_BARRIER(18)
PG_WAIT_BARRIER(19)
PG_WAIT_BARRIER(20)
PG_WAIT_BARRIER(21)
PG_WAIT_BARRIER(22)
PG_WAIT_BARRIER(23)
PG_WAIT_BARRIER(24)
PG_WAIT_BARRIER(25)
PG_WAIT_BARRIER(26)
PG_WAIT_BARRIER(27)
PG_WAIT_BARRIER(28)
PG_WAIT_BARRIER(29)
PG_WAIT_BARRIER(30)
PG_WAIT_BARRIER(31)
PG_WAIT_BARRIER(32)
PG_WAIT_BARRIER(33)
PG_WAIT_BARRIER(34)
PG_WAIT_BARRIER(35)
PG_WAIT_BARRIER(36)
PG_WAIT_BARRIER(37)
PG_WAIT_BARRIER(38)
PG_WAIT_BARRIER(39)
PG_WAIT_BARRIER(40)
PG_WAIT_BARRIER(41)
PG_WAIT_BARRIER(42)
PG_WAIT_BARRIER(43)
PG_WAIT_BARRIER(44)
PG_WAIT_BARRIER(45)
PG_WAIT_BARRIER(46)
PG_WAIT_BARRIER(47)
PG_WAIT_BARRIER(48)
PG_WAIT_BARRIER(49)
PG_WAIT_BARRIER(50)
PG_WAIT_BARRIER(51)
PG_WAIT_BARRIER(52)
PG_WAIT_BARRIER(53)
PG_WAIT_BARRIER(54)
PG_WAIT_BARRIER(55)
PG_WAIT_BARRIER(56)
PG_WAIT_BARRIER(57)
PG_WAIT_BARRIER(58)
PG_WAIT_BARRIER(59)
PG_WAIT_BARRIER(60)
PG_WAIT_BARRIER(61)
PG_WAIT_BARRIER(62)
PG_WAIT_BARRIER(63)
#undef PG_WAIT_BARRIER

// Runtime form of wait_barrier for the ring's drain (n = 0 .. 4 steps of
// L loads each may stay in flight; the counter's limit of 63 only makes the
// wait stricter).
constexpr int vm_cap(int n) { return n < 63 ? n : 63; }
template <int L>
PG_DEV void wait_barrier_steps(int n) {
  switch (n) {
    case 0: wait_barrier<0>(); break;
    case 1: wait_barrier<vm_cap(L)>(); break;
    case 2: wait_barrier<vm_cap(2 * L)>(); break;
    case 3: wait_barrier<vm_cap(3 * L)>(); break;
    default: wait_barrier<vm_cap(4 * L)>(); break;
  }
}

}  // namespace pg
