// Shared device types and helpers for the gfx950 (CDNA4) kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define CRF_DEV __device__ __forceinline__

// Device error flag bits (mirrors crf_context_device_errors).
enum { CRF_DEVERR_BLOCK_TABLE = 1 };

CRF_DEV float bf2f(bf16 x) { return (float)x; }
CRF_DEV bf16 f2bf(float x) { return (bf16)x; }  // round-to-nearest-even on gfx950

CRF_DEV bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }
CRF_DEV u32x4 as_u32x4(bf16x8 v) { return __builtin_bit_cast(u32x4, v); }

CRF_DEV u32x4 ld16(const void *p) { return *reinterpret_cast<const u32x4 *>(p); }
CRF_DEV void st16(void *p, u32x4 v) { *reinterpret_cast<u32x4 *>(p) = v; }
CRF_DEV u32x2 ld8(const void *p) { return *reinterpret_cast<const u32x2 *>(p); }
CRF_DEV void st8(void *p, u32x2 v) { *reinterpret_cast<u32x2 *>(p) = v; }

// the 4 bf16 values of an 8-byte load as floats
CRF_DEV f32x4 unpack_bf16x4(u32x2 v) {
  return f32x4{__builtin_bit_cast(float, v[0] << 16), __builtin_bit_cast(float, v[0] & 0xffff0000u),
               __builtin_bit_cast(float, v[1] << 16), __builtin_bit_cast(float, v[1] & 0xffff0000u)};
}
CRF_DEV u32x2 pack_bf16x4(float a, float b, float c, float d) {
  bf16x4 v = {f2bf(a), f2bf(b), f2bf(c), f2bf(d)};
  return __builtin_bit_cast(u32x2, v);
}

// D[32x32] += A[32x16] * B[16x32]; lane l holds A row l%32 / B column l%32 with
// k = 8*(l/32) .. +8; D element (row 8*(v/4) + 4*(l/32) + v%4, column l%32) in v.
CRF_DEV f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
// D[16x16] += A[16x32] * B[32x16]; lane l holds A row l%16 / B column l%16 with
// k = 8*(l/16) .. +8; D element (row 4*(l/16) + v, column l%16) in v.
CRF_DEV f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Raw buffer resource over [base, base + bytes): loads at or past `bytes`
// return zero (the hardware range check), which is how masked rows are
// zero-filled without branches.
CRF_DEV __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}
CRF_DEV u32x4 bld16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}
constexpr uint32_t CRF_OOB = 0x80000000u;  // any offset >= this is outside every resource we build

// 16-byte-per-lane DMA from a buffer resource straight into LDS: lane L's bytes
// land at lds + 16 L (lds must be wave-uniform).
typedef __attribute__((address_space(3))) char lds_char;
CRF_DEV void dma16(__amdgpu_buffer_rsrc_t r, lds_char *lds, uint32_t voff, uint32_t soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void *)lds, 16, voff, soff, 0, 0);
}

CRF_DEV float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
CRF_DEV float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Workgroups are dispatched round-robin over the 8 XCDs (workgroup i runs on
// XCD i % 8).  Remap so that each XCD receives a contiguous range of logical
// tile indices, which then share operand panels in that XCD's L2.
CRF_DEV int xcd_remap(int bid, int nblocks) {
  const int nx = 8;
  if (nblocks % nx != 0) return bid;
  return (bid % nx) * (nblocks / nx) + bid / nx;
}

// Paged KV cache addressing: element offset of (token, kv_head) row start in a
// layer's pool, or -1 when the block table entry is out of range.
struct PagedKV {
  char *k;        // layer base of the K pool (element type decided by the kernel)
  char *v;
  int64_t page_stride;  // elements
  const int32_t *block_table;
  int n_pages, page_size, n_tokens;
  int *err;
};

CRF_DEV int64_t paged_row(const PagedKV &kv, int token, int kvh, int hd) {
  const int page = kv.block_table[token / kv.page_size];
  if (page < 0 || page >= kv.n_pages) {
    atomicOr(kv.err, (int)CRF_DEVERR_BLOCK_TABLE);
    return -1;
  }
  const int slot = token % kv.page_size;
  return (int64_t)page * kv.page_stride + ((int64_t)kvh * kv.page_size + slot) * hd;
}
