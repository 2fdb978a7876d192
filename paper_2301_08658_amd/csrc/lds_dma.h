// Direct-to-LDS copies for gfx950 kernels (buffer_load_dwordx4 ... lds).
//
// The copies are issued from inline assembly so that the compiler does not
// track them: it would otherwise make every LDS read that it cannot prove
// disjoint from a copy in flight (transposing reads among them) wait for all
// copies (s_waitcnt vmcnt(0)), serializing a copy ring.  Kernels that use
// them order copies and reads themselves (vmcnt waits and barriers).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace atp {
namespace dma {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr uint32_t kRsrcWord3 = 0x00020000u;   // raw 32-bit buffer access
constexpr uint32_t kOob = 0x80000000u;          // offset beyond any num_records

// Buffer resource words for `bytes` bytes from `base` (offsets at or past
// the end read zeros; capped so offsets and sizes stay in 31 bits).
__device__ __forceinline__ u32x4 rsrc_words(const void* base, int64_t bytes) {
    const int64_t cap = 0x7fffff00;
    const uint32_t n = (uint32_t)(bytes < 0 ? 0 : (bytes > cap ? cap : bytes));
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    return u32x4{(uint32_t)a, (uint32_t)(a >> 32) & 0xffffu, n, kRsrcWord3};
}

// One 64-lane copy instruction: lane l's 16 bytes at base + voff (+ soff)
// land in LDS at lds_dst + 16 l.  Only voff is checked against the range.
// The LDS address travels in M0.  The compiler treats M0 as reserved and
// warns that the clobber below is not honoured, i.e. it would not reload a
// value of its own after this statement.  The kernels calling this keep
// nothing in M0 (no LDS-DMA builtins, no indexed register moves, every loop
// over registers unrolled); a kernel that needs M0 itself must not use it.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"   // the M0 clobber, see above
__device__ __forceinline__ void lds_dma16(const u32x4& rs, const uint16_t* lds_dst, uint32_t voff,
                                          uint32_t soff) {
    typedef __attribute__((address_space(3))) const void* lds_cptr;
    const uint32_t m = (uint32_t)(uintptr_t)(lds_cptr)lds_dst;   // LDS byte address
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                 :: "s"(m), "v"(voff), "s"(rs), "s"(soff) : "memory", "m0");
}
#pragma clang diagnostic pop

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

}  // namespace dma
}  // namespace atp
