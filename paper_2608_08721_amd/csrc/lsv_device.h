// Internal device helpers shared by the gfx950 kernels of liblsv.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

// Global-memory view of a pointer.  Pointers reaching a kernel inside a struct are
// generic; generic (flat) accesses also count against the LDS wait counter, which
// forces full waits between the weight stream and LDS reads.  GL() makes every
// global access a global_load / global_store.
#define GL(p) ((__attribute__((address_space(1))) std::remove_reference_t<decltype(*(p))>*)(p))

#define LSV_DEV __device__ __forceinline__

typedef uint16_t bf16_t;  // storage type: IEEE bfloat16 bit pattern
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));  // 16-byte global / LDS accesses
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
#define GLOBAL __attribute__((address_space(1)))

namespace lsv {

constexpr int kWave = 64;

// Streams read once per verify step -- packed weights, the KV cache -- are loaded non-temporal
// (the nt cache policy; for buffer loads, bit 1 of the aux operand): without it these lines are
// cached on their way in, evicting what is re-read (activation fragments) for nothing.  Measured
// on Llama-3-70B at 16 rows: gate/up 150.4 -> 137.2 us per launch, QKV 33.8 -> 31.5.  The scope
// bits (sc0, sc1) on top of nt changed nothing.
constexpr int kBufferStream = 2;

// A raw buffer resource over `bytes` bytes at p (below 4 GiB: the library refuses larger
// packed matrices); loads past the end return zero.
LSV_DEV __amdgpu_buffer_rsrc_t stream_rsrc(const void* p, size_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, (int)(uint32_t)bytes, 0x00020000);
}
// 16 bytes at byte offset `off` of a read-once stream.  A buffer load takes its base from scalar
// registers and one 32-bit lane offset, where a global load needs a 64-bit address per lane
// (Llama-3-70B, lab: down at 36 rows 108.9 -> 100.2 us, O 34.0 -> 31.7, against global nt loads).
LSV_DEV u32x4_t load_stream(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, kBufferStream));
}
// The same through a global address (the batched GEMM body, where buffer loads lost 0.3%).
template <typename T> LSV_DEV T load_stream(const GLOBAL T* p) { return __builtin_nontemporal_load(p); }

LSV_DEV float bf2f(bf16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// fp32 -> bf16, round to nearest even; NaN stays a quiet NaN.
LSV_DEV bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return (bf16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

// Element conversions for the two storage types.
template <typename T> LSV_DEV float to_f32(T x);
template <> LSV_DEV float to_f32<float>(float x) { return x; }
template <> LSV_DEV float to_f32<bf16_t>(bf16_t x) { return bf2f(x); }
template <typename T> LSV_DEV T from_f32(float x);
template <> LSV_DEV float from_f32<float>(float x) { return x; }
template <> LSV_DEV bf16_t from_f32<bf16_t>(float x) { return f2bf(x); }

// Sequence that owns block row m (linear scan: batches are small).
LSV_DEV int seq_of_row(const int32_t* row_offsets, int batch, int m) {
  int b = 0;
  while (b + 1 < batch && GL(row_offsets)[b + 1] <= m) ++b;
  return b;
}

// Device-scope release/acquire around a "last workgroup finishes" counter.
// Returns true in every thread of the workgroup that arrived last.
LSV_DEV bool arrive_last(int* counter, int expected, int* lds_flag) {
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) {
    int old = __hip_atomic_fetch_add(counter, 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    *lds_flag = (old == expected - 1);
  }
  __syncthreads();
  bool last = *lds_flag != 0;
  if (last) __threadfence();
  return last;
}

LSV_DEV void reset_counter(int* counter) {
  if (threadIdx.x == 0) __hip_atomic_store(counter, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

LSV_DEV float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}
LSV_DEV float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

}  // namespace lsv
