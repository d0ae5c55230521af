// The filter test of Sec. 3 stage 3 on one tile of 16-byte vectors held in
// registers, shared by the vector and per-row filter kernels.
//
// Survival test on a transformed word: for a threshold whose pattern is
// non-negative, key(x) >= key(tau) iff bits(x) >= bits(tau) as signed
// integers; for a negative one, iff bits(x) <= bits(tau) as unsigned, which
// is the signed test on bits ^ 0x7FFFFFFF.  So every element costs one XOR
// and one signed compare (bf16: the same per 16-bit half, two per word).
#pragma once

#include <climits>

#include "device_common.h"

namespace profk {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef short s16x2 __attribute__((ext_vector_type(2)));

template <int DT> struct Elem;
template <> struct Elem<0> { static constexpr int EPV = 4, ES = 4, KEYBITS = 32; };
template <> struct Elem<1> { static constexpr int EPV = 8, ES = 2, KEYBITS = 16; };

// The transformed threshold of a key: survive iff transform(word) >= thr.
// Under the lexicographic rule an element equal to the threshold survives
// only when its index is at most `tie` (0xFFFFFFFF: every tie survives, the
// paper's rule); the fast test below stays the superset key >= tau.
template <int DT>
struct Thresh {
  uint32_t flip;
  int thr;
  uint32_t neutral;  // a word that fails the fast test unless every word passes
  uint32_t tie;
  __device__ __forceinline__ bool keep(int x, uint32_t i) const { return x >= thr && (x != thr || i <= tie); }
  __device__ __forceinline__ explicit Thresh(uint32_t tau, uint32_t tie_idx = 0xFFFFFFFFu) : tie(tie_idx) {
    if (DT == 0) {
      const uint32_t tb = bits_from_key_f32(tau);
      flip = (tb >> 31) ? 0x7FFFFFFFu : 0u;
      thr = static_cast<int>(tb ^ flip);
      neutral = 0x80000000u ^ flip;
    } else {
      const uint32_t tb = bits_from_key_bf16(tau);
      const uint32_t f16 = (tb & 0x8000u) ? 0x7FFFu : 0u;
      flip = f16 | (f16 << 16);
      thr = static_cast<int>(static_cast<int16_t>(static_cast<uint16_t>(tb ^ f16)));
      neutral = (0x8000u * 0x10001u) ^ flip;
    }
  }
};

// Fast test: does any element of the lane's tile survive?
template <int DT, int U>
__device__ __forceinline__ bool tile_any(const u32x4 (&v)[U], const Thresh<DT>& th) {
  int mx;
  if (DT == 0) {
    mx = INT_MIN;
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int e = 0; e < 4; ++e) mx = max(mx, static_cast<int>(v[u][e] ^ th.flip));
  } else {
    s16x2 m2 = s16x2{SHRT_MIN, SHRT_MIN};
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int e = 0; e < 4; ++e) m2 = __builtin_elementwise_max(m2, __builtin_bit_cast(s16x2, v[u][e] ^ th.flip));
    mx = max(static_cast<int>(m2.x), static_cast<int>(m2.y));
  }
  return mx >= th.thr;
}

// Exact pass over a lane's tile, taken when some lane of the wave holds a
// survivor.  Vector u of the lane is tile vector vb + u*BS + pos, valid when
// below vend; element e of a vector is input element base + vector*EPV + e.
// The survivor bits of each vector are formed with packed arithmetic: with
// thr1 = thr - 1, the saturating difference thr1 - w is negative iff
// w >= thr, so its sign bits are the survivor flags (bf16: two per word,
// gathered into one mask per vector with byte permutes).  emit() then visits
// each lane's set bits in a short loop per vector instead of one predicated
// branch per element, which matters where survivors are common (a row of the
// per-row path keeps about M/D of its elements, 0.5 % of a 131072-wide bf16
// row, so nearly every wave holds a few in every tile).
// LEX: the lexicographic rule (ties at the threshold cut by index).
template <int DT, int U, int BS, bool LEX = false>
struct TileSparse {
  static constexpr int EPV = Elem<DT>::EPV;
  uint32_t m[U];  // survivor flags of vector u (bit layout: elem_of_bit)
  uint32_t vb, pos, base;

  // bf16 flag bits: element e in 0..3 at bit 8e+7, element e in 4..7 at bit
  // 8(e-4)+6; fp32: element e at bit e.
  static __device__ __forceinline__ uint32_t elem_of_bit(uint32_t p) {
    return DT == 0 ? p : (p >> 3) + ((p & 1u) ? 0u : 4u);
  }

  __device__ __forceinline__ TileSparse(const u32x4 (&v)[U], const Thresh<DT>& th, uint32_t vb_,
                                        uint32_t vend, uint32_t pos_, uint32_t base_)
      : vb(vb_), pos(pos_), base(base_) {
    constexpr uint32_t kAll = DT == 0 ? 0xFu : 0xC0C0C0C0u;
    const bool all = DT == 0 ? th.thr == INT_MIN : th.thr == SHRT_MIN;  // every key survives
#pragma unroll
    for (int u = 0; u < U; ++u) {
      uint32_t b;
      if (DT == 0) {
        const int thr1 = th.thr - (all ? 0 : 1);
        b = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int d = __builtin_elementwise_sub_sat(thr1, static_cast<int>(v[u][e] ^ th.flip));
          b |= (static_cast<uint32_t>(d) >> 31) << e;
        }
      } else {
        const short t1 = static_cast<short>(th.thr - (all ? 0 : 1));
        const s16x2 thr1 = s16x2{t1, t1};
        uint32_t d[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          d[e] = __builtin_bit_cast(uint32_t, __builtin_elementwise_sub_sat(
                                                   thr1, __builtin_bit_cast(s16x2, v[u][e] ^ th.flip)));
        b = (__builtin_amdgcn_perm(d[1], d[0], 0x07050301u) & 0x80808080u) |
            ((__builtin_amdgcn_perm(d[3], d[2], 0x07050301u) >> 1) & 0x40404040u);
      }
      if (all) b = kAll;
      m[u] = vb + u * BS + pos < vend ? b : 0u;
    }
    if (LEX && th.tie != 0xFFFFFFFFu) {
      // lexicographic rule: drop the survivors equal to the threshold whose
      // index lies past the threshold pair's
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const uint32_t i0 = base + (vb + u * BS + pos) * EPV;
        uint32_t b = m[u], keep = m[u];
        while (b) {
          const uint32_t p = __builtin_ctz(b);
          b &= b - 1;
          const uint32_t e = elem_of_bit(p);
          int x;
          if (DT == 0) {
            const uint32_t raw = (e & 2) ? ((e & 1) ? v[u][3] : v[u][2]) : ((e & 1) ? v[u][1] : v[u][0]);
            x = static_cast<int>(raw ^ th.flip);
          } else {
            const uint32_t raw = (e & 4) ? ((e & 2) ? v[u][3] : v[u][2]) : ((e & 2) ? v[u][1] : v[u][0]);
            const uint32_t w = raw ^ th.flip;
            x = (e & 1) ? (static_cast<int>(w) >> 16) : (static_cast<int>(w << 16) >> 16);
          }
          if (!th.keep(x, i0 + e)) keep &= ~(1u << p);
        }
        m[u] = keep;
      }
    }
  }

  __device__ __forceinline__ bool any() const {
    uint32_t o = 0;
#pragma unroll
    for (int u = 0; u < U; ++u) o |= m[u];
    return o != 0;
  }

  __device__ __forceinline__ uint32_t count() const {
    uint32_t c = 0;
#pragma unroll
    for (int u = 0; u < U; ++u) c += __popc(m[u]);
    return c;
  }

  // f(key, index) for each survivor (in flag-bit order within a vector).
  template <class F>
  __device__ __forceinline__ void emit(const u32x4 (&v)[U], F f) const {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t vi = vb + u * BS + pos;
      uint32_t b = m[u];
      while (b) {
        const uint32_t e = elem_of_bit(__builtin_ctz(b));
        b &= b - 1;
        if (DT == 0) {
          const uint32_t raw = (e & 2) ? ((e & 1) ? v[u][3] : v[u][2]) : ((e & 1) ? v[u][1] : v[u][0]);
          f(key_f32(raw), base + vi * EPV + e);
        } else {
          const uint32_t raw = (e & 4) ? ((e & 2) ? v[u][3] : v[u][2]) : ((e & 2) ? v[u][1] : v[u][0]);
          f(key_bf16((e & 1) ? raw >> 16 : raw & 0xFFFFu), base + vi * EPV + e);
        }
      }
    }
  }
};

}  // namespace profk
