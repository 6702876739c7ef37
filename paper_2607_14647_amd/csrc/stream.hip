// Measurement aid: the HBM -> LDS stream rate the verify-step kernels are
// bounded by in practice.  Every wave streams its own contiguous range with
// the loads the GEMM and attention kernels use (buffer loads with the LDS
// destination, 16 bytes per lane, 1 KB per instruction), keeping eight of them
// in flight, into a private LDS ring; nothing is written to memory.  The loads
// are non-temporal (cache policy nt), as the attention's cache stream is: that
// policy streams read-once data faster than the default one.  The published
// 8 TB/s of HBM3E is the roofline peak; this rate, measured with every CU
// streaming, is the attainable one for kernels that stream through LDS.

#include "dcut_internal.h"

namespace dcut {
namespace {

constexpr int SWAVES = 4, SDEPTH = 8;

__global__ void __launch_bounds__(SWAVES * 64)
k_stream(const unsigned char *__restrict__ src, int per_wave) {
  __shared__ __align__(16) unsigned char ring[SWAVES][SDEPTH][1024];
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const unsigned char *base = src + ((long long)blockIdx.x * SWAVES + wave) * per_wave;
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc((void *)base, (short)0, per_wave, 0x00020000);
  const int n = per_wave / 1024;
  for (int i = 0; i < n; ++i) {
    // at most SDEPTH - 1 older loads outstanding before the next slot is refilled
    if (i >= SDEPTH) asm volatile("s_waitcnt vmcnt(7)" ::: "memory");
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void *)&ring[wave][i % SDEPTH][0],
                                             16, (unsigned)(lane * 16), i * 1024, 0, CPOL_NT);
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

}  // namespace
}  // namespace dcut

using namespace dcut;

extern "C" int dcut_stream_probe(const void *src, size_t bytes, int workgroups, hipStream_t stream) {
  if (!src || ((uintptr_t)src & 15) || workgroups < 1 || workgroups > 65536) return DCUT_EINVAL;
  const size_t waves = (size_t)workgroups * SWAVES;
  if (bytes == 0 || bytes % (waves * 1024)) return DCUT_EINVAL;
  const size_t per_wave = bytes / waves;
  if (per_wave > 0x7fffffffu - 1024) return DCUT_EUNSUPPORTED;
  return launch(DCUT_KERNEL_NONE, k_stream, dim3((unsigned)workgroups), dim3(SWAVES * 64), 0, stream,
                (const unsigned char *)src, (int)per_wave);
}
