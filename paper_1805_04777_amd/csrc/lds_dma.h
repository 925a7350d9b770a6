// lds_dma.h -- buffer loads that write straight into LDS (gfx950), shared by
// the HIP translation units of libconvcrf.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>

namespace convcrf {

// s_waitcnt operand that waits until at most n vector-memory operations of
// the wave are outstanding (gfx9 encoding; expcnt and lgkmcnt untouched).
constexpr int vm_wait(int n) {
    const int v = n < 0 ? 0 : (n > 63 ? 63 : n);
    return (v & 15) | (v >> 4) << 14 | 7 << 4 | 15 << 8;
}

// One 64-lane buffer load into LDS: lane l writes the dword at byte offset
// voffset + soffset of the buffer (zero when out of range) to LDS byte
// lds_base + 4 l.  Written as assembly so that the compiler neither counts
// it nor waits for it before LDS reads of other rows: the caller waits with
// an explicit vmcnt and a work-group barrier before reading what it wrote.
typedef int rsrc_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void lds_dma(rsrc_t rsrc, unsigned voffset, int soffset,
                                        unsigned lds_base) {
    asm volatile("s_mov_b32 m0, %3\n\ts_nop 0\n\tbuffer_load_dword %0, %1, %2 offen lds"
                 :
                 : "v"(voffset), "s"(rsrc), "s"(soffset), "s"(lds_base)
                 : "memory", "m0");
}

// The same with 16 bytes per lane (LDS byte lds_base + 16 l); voffset and
// soffset must be multiples of 16.
__device__ __forceinline__ void lds_dma16(rsrc_t rsrc, unsigned voffset, int soffset,
                                          unsigned lds_base) {
    asm volatile("s_mov_b32 m0, %3\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds"
                 :
                 : "v"(voffset), "s"(rsrc), "s"(soffset), "s"(lds_base)
                 : "memory", "m0");
}

__device__ __forceinline__ rsrc_t buffer_rsrc(const float* base, unsigned bytes) {
    const unsigned long long p = reinterpret_cast<unsigned long long>(base);
    rsrc_t r;
    r.x = (int)(unsigned)p;
    r.y = (int)(unsigned)(p >> 32);            // stride 0
    r.z = (int)bytes;                           // num_records
    r.w = 0x00020000;                           // raw dword access
    return r;
}

// Buffer offset past any buffer of under 2 GB: the load reads zero.
constexpr unsigned kDmaOob = 0x80000000u;

}  // namespace convcrf
