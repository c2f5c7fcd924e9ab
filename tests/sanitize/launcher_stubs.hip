// Stand-ins for the library's kernel launchers, for the host-only sanitizer
// build of the C ABI: every launcher fails without touching its arguments,
// so the build links without any kernel and can never enqueue one.
#include "../../paper_2609_35139_amd/csrc/launch.h"

namespace cr {

hipError_t copy_table(const int32_t*, int, int*, hipStream_t) { return hipErrorInvalidValue; }
hipError_t chunk_schedule(const int32_t*, int32_t, const int32_t*, int32_t, int, const int32_t*,
                          int*, int*, int*, int*, int*, hipStream_t, float2*, int, double) {
  return hipErrorInvalidValue;
}
hipError_t key_rope_table(float2*, const int*, int, const KeyRope&, hipStream_t) {
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t gemm_bias(const T*, int64_t, const T*, int64_t, int, int, int, T*, int64_t,
                     const float*, const T*, int64_t, bool, hipStream_t, const T*, int64_t) {
  return hipErrorInvalidValue;
}
template <typename T>
hipError_t gemm_bias_split(const T*, int64_t, int, const T*, int64_t, const T*, int64_t, int, int,
                           int, T*, int64_t, const float*, const T*, int64_t, hipStream_t) {
  return hipErrorInvalidValue;
}
template <typename T>
hipError_t compose_bias(const T*, const T*, int64_t, const T*, const T*, float*, int, int,
                        hipStream_t) {
  return hipErrorInvalidValue;
}
template <typename T>
hipError_t transpose_into(const T*, const T*, T*, int64_t, int, int, hipStream_t) {
  return hipErrorInvalidValue;
}
template <typename T>
hipError_t gemm_qkv(const T*, int64_t, const T*, int, int, int, int, T*, T*, T*, int64_t,
                    const float*, const float2*, hipStream_t) {
  return hipErrorInvalidValue;
}
template <typename T>
hipError_t gemm_expand(const T*, int64_t, const T*, int, int, int, T*, KvStrides, const float*,
                       const float*, int, const int*, const float2*, T*, KvStrides, hipStream_t) {
  return hipErrorInvalidValue;
}
template <typename T>
hipError_t attention(const T*, const T*, const T*, T*, int, int, int, int, int64_t, const int*,
                     const int*, hipStream_t) {
  return hipErrorInvalidValue;
}
template <typename T>
hipError_t layernorm(const T*, int64_t, T*, int64_t, const float*, const float*, int, int, float,
                     hipStream_t) {
  return hipErrorInvalidValue;
}
template <typename T>
hipError_t compress_segments(const T*, KvStrides, int, const T*, const float*, T*, int64_t, int,
                             int, hipStream_t) {
  return hipErrorInvalidValue;
}
template <typename T>
hipError_t rotate_keys(T*, KvStrides, int, int, const float2*, bool, float, hipStream_t) {
  return hipErrorInvalidValue;
}
template <typename Tin, typename Tout>
hipError_t transpose_convert(const Tin*, Tout*, int, int, int, int, int64_t, const float*,
                             hipStream_t) {
  return hipErrorInvalidValue;
}
template <typename Tin>
hipError_t convert_f32(const Tin*, float*, int64_t, int64_t, int, int64_t, int64_t, hipStream_t) {
  return hipErrorInvalidValue;
}

#define STUBS(T)                                                                                  \
  template hipError_t gemm_bias<T>(const T*, int64_t, const T*, int64_t, int, int, int, T*,      \
                                   int64_t, const float*, const T*, int64_t, bool, hipStream_t,   \
                                   const T*, int64_t);                                            \
  template hipError_t gemm_bias_split<T>(const T*, int64_t, int, const T*, int64_t, const T*,   \
                                         int64_t, int, int, int, T*, int64_t, const float*,      \
                                         const T*, int64_t, hipStream_t);                        \
  template hipError_t compose_bias<T>(const T*, const T*, int64_t, const T*, const T*, float*,  \
                                      int, int, hipStream_t);                                    \
  template hipError_t transpose_into<T>(const T*, const T*, T*, int64_t, int, int, hipStream_t); \
  template hipError_t gemm_qkv<T>(const T*, int64_t, const T*, int, int, int, int, T*, T*, T*,   \
                                  int64_t, const float*, const float2*, hipStream_t);             \
  template hipError_t gemm_expand<T>(const T*, int64_t, const T*, int, int, int, T*, KvStrides,   \
                                     const float*, const float*, int, const int*, const float2*,  \
                                     T*, KvStrides, hipStream_t);                                 \
  template hipError_t attention<T>(const T*, const T*, const T*, T*, int, int, int, int, int64_t, \
                                   const int*, const int*, hipStream_t);                          \
  template hipError_t layernorm<T>(const T*, int64_t, T*, int64_t, const float*, const float*,   \
                                   int, int, float, hipStream_t);                                 \
  template hipError_t compress_segments<T>(const T*, KvStrides, int, const T*, const float*, T*, \
                                           int64_t, int, int, hipStream_t);                       \
  template hipError_t rotate_keys<T>(T*, KvStrides, int, int, const float2*, bool, float,        \
                                     hipStream_t);                                                \
  template hipError_t transpose_convert<T, T>(const T*, T*, int, int, int, int, int64_t,         \
                                              const float*, hipStream_t);                         \
  template hipError_t convert_f32<T>(const T*, float*, int64_t, int64_t, int, int64_t, int64_t,  \
                                     hipStream_t);
STUBS(bf16)
STUBS(float)
#undef STUBS

}  // namespace cr
