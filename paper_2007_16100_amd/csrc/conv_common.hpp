// conv_common.hpp -- helpers shared by the sparse-convolution kernels
// (conv.hip: plan, tile and vector-ALU kernels; conv_union.hip: the 3x3x3
// neighbour-table kernel).
#pragma once

#include "spv_internal.hpp"

namespace spv {

constexpr int kChunk = 16;  // rows / pairs per MFMA N-tile
constexpr int kMaxK3 = 27;

__device__ inline int64_t clamp_rows(const int64_t* d, int64_t cap) {
    if (!d) return cap;
    int64_t c = *d;
    return c < 0 ? 0 : (c > cap ? cap : c);
}

constexpr uint32_t kOutOfRange = 0xFFFFF000u;  // a buffer offset past every record

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x2 __attribute__((ext_vector_type(2)));

__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}

// byte address of an LDS location (what M0 takes)
__device__ inline uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// 64 lanes x 16 bytes from gbase + voff -> LDS at lds (asynchronous, counted in vmcnt)
__device__ inline void lds_dma_x4(uint64_t gbase, uint32_t voff, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
                 :
                 : "v"(voff), "s"(gbase), "s"(lds)
                 : "memory", "m0");
}

// wait until at most N vector-memory loads are outstanding
template <int N>
__device__ inline void vm_wait() {
    asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}
__device__ inline void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" : : : "memory"); }


// the 3x3x3 neighbour-table kernel (conv_union.hip)
bool union_supported(int K3, int Cin, int Cout, int dt);
void launch_conv_union(hipStream_t s, const ConvPlan& p, const void* in, int Cin, int64_t in_rows, int Cout,
                       const void* wpack, const float* scale, const float* shift, int relu, void* out, int dt);

}  // namespace spv
