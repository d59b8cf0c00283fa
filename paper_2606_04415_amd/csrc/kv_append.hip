// KV append: the write side of the paged KV pool that prefill and decode of
// one device share (Sec. 3.4, "Memory Locality": co-located phases extend and
// read one pool instead of moving KV caches between workers). Each new token's
// key row, and value row unless values alias keys, is copied into its slot
// (page = slot / P, row = slot % P) of the paged caches.
//
// HBM-bound copy: one thread per 16-byte chunk of a token's row, so a wave
// reads 1 KB of consecutive new-token data and writes it to consecutive
// bytes of one cache row (heads of a slot are contiguous when the head stride
// equals the head dimension). Out-of-range slots are skipped and counted.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.h"

namespace flexattn {

namespace {

struct alignas(16) Chunk {
  uint32_t w[4];
};

__global__ __launch_bounds__(256) void kv_append_kernel(AppendParams a) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t per_tok = a.ck + a.cv;   // 16-byte chunks of one token (K then V)
  if (i >= a.n_tokens * per_tok) return;
  const int64_t t = i / per_tok;
  int64_t c = i - t * per_tok;
  const int32_t slot = a.slot_mapping[t];
  if (slot < 0) return;                      // padding token
  if (int64_t(slot) >= a.num_slots) {        // outside the pool: skipped, counted once per token
    if (c == 0 && a.bad_count) atomicAdd(a.bad_count, 1);
    return;
  }
  const int64_t page = slot / a.P, row = slot - page * a.P;
  const bool is_v = c >= a.ck;
  if (is_v) c -= a.ck;
  const int d = is_v ? a.dv : a.dk;
  const int cpd = d / 8;                     // chunks per head
  const int64_t h = c / cpd, x = 8 * (c - h * cpd);
  const uint16_t* src = (is_v ? a.v_new + t * a.v_new_stride : a.k_new + t * a.k_new_stride) + h * d + x;
  const CacheRef& dst_ref = is_v ? a.vc : a.kc;
  uint16_t* dst = const_cast<uint16_t*>(dst_ref.base) + page * dst_ref.sp + row * dst_ref.ss + h * dst_ref.sh + x;
  *reinterpret_cast<Chunk*>(dst) = *reinterpret_cast<const Chunk*>(src);
}

}  // namespace

hipError_t launch_kv_append(const AppendParams& a, hipStream_t stream) {
  const int64_t total = a.n_tokens * (a.ck + a.cv);
  if (total == 0) return hipSuccess;
  const int64_t blocks = (total + 255) / 256;
  if (blocks > int64_t(INT32_MAX)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(kv_append_kernel, dim3(uint32_t(blocks)), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace flexattn
