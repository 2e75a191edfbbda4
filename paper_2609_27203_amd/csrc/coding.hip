// Column coding of the scalar types that the join kernels do not see as
// they are (the paper's eight-type system, Sec. 3.2 "Type system").  Every
// stored column is four bytes wide and compares as int32, so each type gets
// an order-preserving image in int32:
//   u32       v ^ 0x80000000 (unsigned order becomes signed order);
//   bool      0 or 1 from one byte;
//   i64, u64, f64
//             the rank of the value's total-order key in the context's
//             sorted dictionary of that type (distinct values seen so far):
//             i64 key = bits ^ 2^63, u64 key = bits, f64 key = IEEE 754
//             totalOrder (negative values: all bits flipped; others: the
//             sign bit set).
// Equal images mean identical values and image order is the type's order,
// so joins, comparisons, min/max folds, set deduplication and the canonical
// read order all run unchanged on the images.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/xlh.h"
#include "device_util.h"
#include "kernels.h"

namespace xlh {
namespace k {

constexpr uint32_t U32_BIAS = 0x80000000u;
constexpr u64 SIGN64 = 1ull << 63;

__global__ void encode_narrow_k(const void* in, int ltype, int64_t n, uint32_t* out, uint32_t* bad) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    if (ltype == XL_BOOL) {
      const uint8_t b = ((const uint8_t*)in)[i];
      if (b > 1u) atomicOr(bad, 1u);
      out[i] = b != 0u;
    } else {
      out[i] = ((const uint32_t*)in)[i] ^ U32_BIAS;
    }
  }
}

hipError_t encode_narrow(const void* in, int ltype, int64_t n, uint32_t* out, uint32_t* bad, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  encode_narrow_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(in, ltype, n, out, bad);
  return hipGetLastError();
}

__device__ __forceinline__ u64 order_key(u64 v, int ltype) {
  if (ltype == XL_I64) return v ^ SIGN64;
  if (ltype == XL_F64) return (v & SIGN64) ? ~v : (v | SIGN64);
  return v;  // XL_U64
}

__device__ __forceinline__ u64 from_order_key(u64 k, int ltype) {
  if (ltype == XL_I64) return k ^ SIGN64;
  if (ltype == XL_F64) return (k & SIGN64) ? (k & ~SIGN64) : ~k;
  return k;
}

__global__ void order_keys64_k(const u64* in, int ltype, int64_t n, u64* out) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    out[i] = order_key(in[i], ltype);
}

hipError_t order_keys64(const u64* in, int ltype, int64_t n, u64* out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  order_keys64_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(in, ltype, n, out);
  return hipGetLastError();
}

__global__ void unique_flags64_k(const u64* sorted, int64_t n, uint32_t* flag) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    flag[i] = i == 0 || sorted[i] != sorted[i - 1];
}

hipError_t unique_flags64(const u64* sorted, int64_t n, uint32_t* flag, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  unique_flags64_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(sorted, n, flag);
  return hipGetLastError();
}

__global__ void compact64_k(const u64* src, const uint32_t* flag, const uint32_t* pos, u64* dst, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    if (flag[i]) dst[pos[i]] = src[i];
}

hipError_t compact64(const u64* src, const uint32_t* flag, const uint32_t* pos, u64* dst, int64_t n,
                     hipStream_t s) {
  if (n <= 0) return hipSuccess;
  compact64_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(src, flag, pos, dst, n);
  return hipGetLastError();
}

// out[i] = number of dictionary keys below q[i] (its rank when present).
__global__ void rank64_k(const u64* dict, int64_t nd, const u64* q, int64_t n, uint32_t* out) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const u64 key = q[i];
    int64_t lo = 0, hi = nd;
    while (lo < hi) {
      const int64_t mid = (lo + hi) >> 1;
      if (dict[mid] < key) lo = mid + 1;
      else hi = mid;
    }
    out[i] = (uint32_t)lo;
  }
}

hipError_t rank64(const u64* dict, int64_t nd, const u64* q, int64_t n, uint32_t* out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  rank64_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(dict, nd, q, n, out);
  return hipGetLastError();
}

__global__ void remap_k(uint32_t* col, int64_t n, const uint32_t* map) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    col[i] = map[col[i]];
}

hipError_t remap_codes(uint32_t* col, int64_t n, const uint32_t* map, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  remap_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(col, n, map);
  return hipGetLastError();
}

// Values of the images img[0..n): 1-byte bools, 4-byte u32 or 8-byte
// dictionary values.
__global__ void decode_k(const uint32_t* img, int64_t n, int ltype, const u64* dict, void* out) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t v = img[i];
    if (ltype == XL_BOOL) ((uint8_t*)out)[i] = (uint8_t)v;
    else if (ltype == XL_U32) ((uint32_t*)out)[i] = v ^ U32_BIAS;
    else ((u64*)out)[i] = from_order_key(dict[v], ltype);
  }
}

hipError_t decode_column(const uint32_t* img, int64_t n, int ltype, const u64* dict, void* out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  decode_k<<<grid_for(n, 256, 65536), 256, 0, s>>>(img, n, ltype, dict, out);
  return hipGetLastError();
}

}  // namespace k
}  // namespace xlh
