// Selection helpers shared by the routing kernels: bounded sorted lists of the best (key,
// node) pairs, and the order-preserving map of float bits to unsigned integers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace maestro {

// internal "empty slot" index of a TopK list, reported as -1
constexpr int32_t kNoNode = INT32_MAX;

template <int KT>
struct TopK {
  float s[KT];
  int32_t n[KT];

  __device__ __forceinline__ void init() {
#pragma unroll
    for (int i = 0; i < KT; ++i) { s[i] = INFINITY; n[i] = kNoNode; }
  }
  // Insert a candidate whose node index is larger than every node already held (nodes are
  // visited in increasing order within a lane): equal scores stay behind, so comparing
  // scores strictly gives the lexicographic order.
  __device__ __forceinline__ void push_increasing(float sc, int32_t node) {
    if (!(sc < s[KT - 1])) return;   // cannot enter: the common case once the list is full
#pragma unroll
    for (int i = KT - 1; i >= 0; --i) {
      const int p = i > 0 ? i - 1 : 0;
      const bool lt_prev = (i > 0) && sc < s[p];
      if (sc < s[i]) {
        if (lt_prev) { s[i] = s[p]; n[i] = n[p]; }
        else { s[i] = sc; n[i] = node; }
      }
    }
  }
  // push_increasing for a candidate that may be absent (ok == false): the presence test joins
  // the entry test, so an absent candidate costs no select of its own
  __device__ __forceinline__ void push_increasing_if(bool ok, float sc, int32_t node) {
    if (!(ok && sc < s[KT - 1])) return;
#pragma unroll
    for (int i = KT - 1; i >= 0; --i) {
      const int p = i > 0 ? i - 1 : 0;
      const bool lt_prev = (i > 0) && sc < s[p];
      if (sc < s[i]) {
        if (lt_prev) { s[i] = s[p]; n[i] = n[p]; }
        else { s[i] = sc; n[i] = node; }
      }
    }
  }
  // General lexicographic insertion, for candidates out of node order (lists merged from other
  // lanes, nodes visited late).
  __device__ __forceinline__ void push_lex(float sc, int32_t node) {
    if (!(sc < s[KT - 1] || (sc == s[KT - 1] && node < n[KT - 1]))) return;   // cannot enter
#pragma unroll
    for (int i = KT - 1; i >= 0; --i) {
      const int p = i > 0 ? i - 1 : 0;
      const bool lt_this = sc < s[i] || (sc == s[i] && node < n[i]);
      const bool lt_prev = (i > 0) && (sc < s[p] || (sc == s[p] && node < n[p]));
      if (lt_this) {
        if (lt_prev) { s[i] = s[p]; n[i] = n[p]; }
        else { s[i] = sc; n[i] = node; }
      }
    }
  }
};

template <>
__device__ __forceinline__ void TopK<1>::push_increasing(float sc, int32_t node) {
  if (sc < s[0]) { s[0] = sc; n[0] = node; }
}
template <>
__device__ __forceinline__ void TopK<1>::push_increasing_if(bool ok, float sc, int32_t node) {
  if (ok && sc < s[0]) { s[0] = sc; n[0] = node; }
}

// order-preserving map of float bits to unsigned (a < b <=> map(a) < map(b), -0 < +0)
__device__ __forceinline__ uint32_t float_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_float(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

}  // namespace maestro
