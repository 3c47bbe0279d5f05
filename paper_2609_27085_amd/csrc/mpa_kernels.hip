// HIP kernels for one mixed prefill+decode attention step on gfx950.
//
// Cache layout (X = 16 / element bytes):
//   K  [block][kv_head][d/X][16][X]   -- a 16-byte chunk of one key row is X
//                                       consecutive dims; the 16 slots of a
//                                       block sit side by side per chunk
//   V  [block][kv_head][d][16]         -- each dim row holds the block's 16
//                                       tokens contiguously
// With this layout both MFMA operands that come from the cache load as whole
// 512-1024 byte runs per wave instruction, in exactly the register layout the
// matrix cores want, with no shuffles:
//
//   S^T[key][row] = K[key][:] . Q^T[:][row]       (A = K chunks, B = Q chunks)
//   O^T[dim][row] = V^T[dim][key] . P^T[key][row] (A = V^T, B = P from S^T)
//
// In the 16x16 MFMA output a lane holds 4 consecutive rows of one column, so
// lane (n, g) of a wave owns query row n and keys 4g..4g+3 of each 16-key
// block; the softmax state of row n (running max, sum) is lane-local up to a
// 4-way reduction across the lane groups, and P^T is already in B-operand
// order for the PV product.
//
// Softmax runs in base 2: scores are scaled by scale*log2(e), exponentials are
// v_exp_f32, and log-sum-exp values are returned in natural log units.

#include <math.h>
#include <stdint.h>

#include <atomic>

#include "mpa_internal.h"

namespace mpa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// acc + the two bf16 values packed in w (one v_dot2 against (1, 1)); the
// products are exact and the sum is taken in f32
__device__ inline float add_bf16_pair(unsigned w, float acc) {
  const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), one, acc, false);
}

constexpr float kLn2 = 0.69314718055994530942f;

__device__ inline int wave_uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ inline float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// max(x[lane], x[lane ^ 32]) with one VALU lane swap (no LDS round trip, so
// no wait on outstanding LDS reads)
__device__ inline float max_across_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ inline short bf16_bits(float x) { return __builtin_bit_cast(short, (__bf16)x); }

// s_waitcnt immediate that waits until at most n vector-memory operations are
// outstanding (expcnt and lgkmcnt left at their maxima).  Used through the
// intrinsic, which the compiler's own wait-count tracking understands.
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
#define MPA_WAIT_VMCNT(n)                          \
  do {                                             \
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(n));      \
    asm volatile("" ::: "memory");                 \
  } while (0)
// The same for the LDS / scalar-memory counter (vmcnt and expcnt left at
// their maxima).
constexpr int lgkmcnt_imm(int n) { return 15 | (7 << 4) | ((n & 15) << 8) | (3 << 14); }
#define MPA_WAIT_LGKMCNT(n)                        \
  do {                                             \
    __builtin_amdgcn_s_waitcnt(lgkmcnt_imm(n));    \
    asm volatile("" ::: "memory");                 \
  } while (0)

// 16 bytes per lane from global memory straight into LDS: lane l reads the
// 16 bytes at base + voff (base uniform, held in SGPRs; voff the lane's byte
// offset) and they land at lds + 16*l (lds the same for the whole wave).
// With the base in SGPRs the per-lane offsets are loop invariant, so a copy
// needs no per-copy address arithmetic in VGPRs (whose reuse would make each
// copy wait for the previous one to be sent).  Issued as inline assembly so
// that the compiler does not make every later LDS read wait for it (it cannot
// tell that the read targets another buffer); the caller waits with an
// explicit vector-memory wait before the barrier that publishes the tile.  M0
// is written only here in this file.
__device__ inline void global_to_lds16(const void* base, unsigned voff, void* lds) {
  const unsigned off = (unsigned)(size_t)(__attribute__((address_space(3))) void*)lds;
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(base), "s"(off) : "memory");
}
// The same copy as a non-temporal (streaming) load, for data read once.
__device__ inline void global_to_lds16_nt(const void* base, unsigned voff, void* lds) {
  const unsigned off = (unsigned)(size_t)(__attribute__((address_space(3))) void*)lds;
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1 nt" ::"v"(voff), "s"(base), "s"(off) : "memory");
}

// Cache reads on the decode path take non-temporal loads: a decode step
// reads each (block, KV head) granule of K and V once, and marking the loads
// as streaming lifts the sustained read rate of scattered 4 KB granules on
// gfx950 by about a tenth over plain loads (the same holds for contiguous
// streams).
template <typename V>
__device__ inline V ld_stream(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const V*>(p));
}

// ---------------------------------------------------------------------------
// Element-type traits.  A "round" of the QK^T product consumes one 16-byte
// chunk of K and of Q per lane: one 16x16x32 bf16 MFMA, or four 16x16x4 f32
// MFMAs.  The PV product consumes 4 tokens of one V^T row per lane: one
// 16x16x16 bf16 MFMA, or four 16x16x4 f32 MFMAs.
template <int DT>
struct Tr;

template <>
struct Tr<0> {  // bf16
  using Elem = uint16_t;   // cache element
  using QElem = uint16_t;  // queries, new rows and outputs
  static constexpr int X = 8;
  using Chunk = bf16x8;
  using VFrag = s16x4;
  using PFrag = s16x4;
  static __device__ inline Chunk load_chunk(const Elem* p) { return __builtin_bit_cast(Chunk, ld_stream<u32x4>(p)); }
  static __device__ inline Chunk load_q(const QElem* p) { return load_chunk(p); }
  static __device__ inline Chunk zero_chunk() {
    u32x4 z = {0u, 0u, 0u, 0u};
    return __builtin_bit_cast(Chunk, z);
  }
  static __device__ inline f32x4 qk(Chunk k, Chunk q, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(k, q, c, 0, 0, 0);
  }
  static __device__ inline VFrag load_v(const Elem* p) { return __builtin_bit_cast(VFrag, ld_stream<u32x2>(p)); }
  static __device__ inline VFrag keep_first(VFrag v, int nvalid) {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = e < nvalid ? v[e] : (short)0;
    return v;
  }
  static constexpr bool kRoundsP = true;  // the PV product takes P in bf16
  static __device__ inline PFrag make_p(f32x4 p) {
    PFrag r;
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = bf16_bits(p[e]);
    return r;
  }
  // p - hi rounded to bf16: hi + lo carries p to about 16 significant bits
  static __device__ inline PFrag make_p_lo(f32x4 p, PFrag hi) {
    PFrag r;
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = bf16_bits(p[e] - __uint_as_float((unsigned)(uint16_t)hi[e] << 16));
    return r;
  }
  static __device__ inline f32x4 pv(VFrag v, PFrag p, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(v, p, c, 0, 0, 0);
  }
  // acc + the probabilities exactly as the PV product consumes them (after
  // rounding to bf16), so that the softmax denominator matches the numerator
  static __device__ inline float psum(f32x4, PFrag pf, float acc) {
    const u32x2 w = __builtin_bit_cast(u32x2, pf);
    return add_bf16_pair(w[1], add_bf16_pair(w[0], acc));
  }
  static __device__ inline void store4(Elem* dst, f32x4 v) {
    s16x4 r;
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = bf16_bits(v[e]);
    *reinterpret_cast<u32x2*>(dst) = __builtin_bit_cast(u32x2, r);
  }
  static __device__ inline void store1(Elem* dst, float v) { *dst = (uint16_t)bf16_bits(v); }
  static __device__ inline void unpack(u32x4 w, float (&f)[X]) {
#pragma unroll
    for (int e = 0; e < X; ++e) f[e] = __uint_as_float(((w[e / 2] >> (16 * (e & 1))) & 0xFFFFu) << 16);
  }
  static __device__ inline u32x4 pack(const float (&f)[X]) {
    u32x4 w;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = (unsigned)(uint16_t)bf16_bits(f[2 * i]) | ((unsigned)(uint16_t)bf16_bits(f[2 * i + 1]) << 16);
    return w;
  }
};

template <>
struct Tr<1> {  // f32
  using Elem = float;
  using QElem = float;
  static constexpr int X = 4;
  using Chunk = f32x4;
  using VFrag = f32x4;
  using PFrag = f32x4;
  static __device__ inline Chunk load_chunk(const Elem* p) { return ld_stream<f32x4>(p); }
  static __device__ inline Chunk load_q(const QElem* p) { return load_chunk(p); }
  static __device__ inline Chunk zero_chunk() { return f32x4{0.f, 0.f, 0.f, 0.f}; }
  static __device__ inline f32x4 qk(Chunk k, Chunk q, f32x4 c) {
#pragma unroll
    for (int j = 0; j < 4; ++j) c = __builtin_amdgcn_mfma_f32_16x16x4f32(k[j], q[j], c, 0, 0, 0);
    return c;
  }
  static __device__ inline VFrag load_v(const Elem* p) { return ld_stream<f32x4>(p); }
  static __device__ inline VFrag keep_first(VFrag v, int nvalid) {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = e < nvalid ? v[e] : 0.f;
    return v;
  }
  static constexpr bool kRoundsP = false;
  static __device__ inline PFrag make_p(f32x4 p) { return p; }
  static __device__ inline PFrag make_p_lo(f32x4, PFrag) { return f32x4{0.f, 0.f, 0.f, 0.f}; }
  static __device__ inline float psum(f32x4 p, PFrag, float acc) { return acc + ((p[0] + p[1]) + (p[2] + p[3])); }
  static __device__ inline f32x4 pv(VFrag v, PFrag p, f32x4 c) {
#pragma unroll
    for (int j = 0; j < 4; ++j) c = __builtin_amdgcn_mfma_f32_16x16x4f32(v[j], p[j], c, 0, 0, 0);
    return c;
  }
  static __device__ inline void store4(Elem* dst, f32x4 v) { *reinterpret_cast<f32x4*>(dst) = v; }
  static __device__ inline void store1(Elem* dst, float v) { *dst = v; }
  static __device__ inline void unpack(u32x4 w, float (&f)[X]) {
#pragma unroll
    for (int e = 0; e < X; ++e) f[e] = __uint_as_float(w[e]);
  }
  static __device__ inline u32x4 pack(const float (&f)[X]) {
    u32x4 w;
#pragma unroll
    for (int e = 0; e < X; ++e) w[e] = __float_as_uint(f[e]);
    return w;
  }
};

// fp8 caches (OCP E4M3 codes) beside bf16 queries, new rows and outputs.
// Codes become bf16 on load (exact: every E4M3 value is a bf16 value) and
// the arithmetic is the bf16 path's; the tensors' scales are applied outside
// (key scale in the softmax scale, value scale on the outputs).
template <>
struct Tr<2> {
  using Elem = uint8_t;
  using QElem = uint16_t;
  static constexpr int X = 8;  // codes per K chunk: 8 bytes
  using Chunk = bf16x8;
  using VFrag = s16x4;
  using PFrag = s16x4;
  static constexpr bool kRoundsP = true;
  static __device__ inline unsigned cvt2(unsigned w, bool hi) {
    return hi ? __builtin_bit_cast(unsigned, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)w, 1.0f, true))
              : __builtin_bit_cast(unsigned, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)w, 1.0f, false));
  }
  static __device__ inline Chunk k_from_codes(u32x2 w) {
    const u32x4 r = {cvt2(w[0], false), cvt2(w[0], true), cvt2(w[1], false), cvt2(w[1], true)};
    return __builtin_bit_cast(Chunk, r);
  }
  static __device__ inline VFrag v_from_codes(unsigned w) {
    const u32x2 r = {cvt2(w, false), cvt2(w, true)};
    return __builtin_bit_cast(VFrag, r);
  }
  static __device__ inline Chunk load_chunk(const Elem* p) { return k_from_codes(ld_stream<u32x2>(p)); }
  static __device__ inline Chunk load_q(const QElem* p) { return Tr<0>::load_q(p); }
  static __device__ inline Chunk zero_chunk() { return Tr<0>::zero_chunk(); }
  static __device__ inline f32x4 qk(Chunk k, Chunk q, f32x4 c) { return Tr<0>::qk(k, q, c); }
  static __device__ inline VFrag load_v(const Elem* p) { return v_from_codes(ld_stream<unsigned>(p)); }
  static __device__ inline VFrag keep_first(VFrag v, int nvalid) { return Tr<0>::keep_first(v, nvalid); }
  static __device__ inline PFrag make_p(f32x4 p) { return Tr<0>::make_p(p); }
  static __device__ inline PFrag make_p_lo(f32x4 p, PFrag hi) { return Tr<0>::make_p_lo(p, hi); }
  static __device__ inline f32x4 pv(VFrag v, PFrag p, f32x4 c) { return Tr<0>::pv(v, p, c); }
  static __device__ inline float psum(f32x4 p, PFrag pf, float acc) { return Tr<0>::psum(p, pf, acc); }
  static __device__ inline void store4(QElem* dst, f32x4 v) { Tr<0>::store4(dst, v); }
  static __device__ inline void store1(QElem* dst, float v) { Tr<0>::store1(dst, v); }
};

// float32 -> OCP E4M3 code: round to nearest, ties to the even mantissa;
// magnitudes from 464 up (which would round past the largest finite value,
// 448) saturate to 448; NaN -> the NaN code; the sign is kept.
__device__ inline unsigned f32_to_e4m3(float x) {
  const unsigned u = __float_as_uint(x);
  const unsigned sign = (u >> 24) & 0x80u;
  const float a = fabsf(x);
  if (a != a) return sign | 0x7Fu;
  if (a >= 464.f) return sign | 0x7Eu;
  if (a < 0.015625f) return sign | (unsigned)rintf(a * 512.f);  // subnormals m * 2^-9 (8 = 2^-6)
  unsigned ua = __float_as_uint(a);
  ua += 0x7FFFFu + ((ua >> 20) & 1u);  // round the f32 mantissa to 3 bits, ties to even
  return sign | ((((ua >> 23) - 120u) << 3) | ((ua >> 20) & 7u));
}

// Largest j in [0, n) with starts[j] <= x (starts non-decreasing, starts[0] <= x).
__device__ inline int upper_index(const int32_t* starts, int n, int x) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (starts[mid] <= x) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// ---------------------------------------------------------------------------
// One wave's online-softmax attention of 16 query rows (one per lane column
// n) against cache blocks kb_begin .. kb_end-1 of one sequence and KV head.
// Key `key` is visible to row n iff key <= limit (per lane) and key < kend;
// V rows of keys >= kend are replaced by zero (they may hold NaN/Inf).
//
// The loop is software-pipelined one block deep: block kb+1's K and V
// fragments are in flight while block kb is consumed.  Block ids come from a
// coalesced load of up to 64 consecutive block-table entries, one per lane,
// and are broadcast with readlane.
template <int DT, int D>
struct RowState {
  f32x4 acc[D / 16];
  float m;  // reference maximum of the row's scaled scores (log2 units)
  float l;  // this lane's part of the running sum of 2^(s*c - m), as rounded for the PV product
};

template <int DT, int D>
struct BlockFrags {
  typename Tr<DT>::Chunk k[D / (4 * Tr<DT>::X)];
  typename Tr<DT>::VFrag v[D / 16];
};

template <int DT, int D>
__device__ inline void load_block(const AttnArgs& a, int blk, int g, BlockFrags<DT, D>& f) {
  using T = Tr<DT>;
  using E = typename T::Elem;
  constexpr int X = T::X;
  const int lane = threadIdx.x & 63;
  const int n = lane & 15, grp = lane >> 4;
  const size_t base = ((size_t)blk * a.hkv + g) * ((size_t)D * kBlock);
  const E* kp = reinterpret_cast<const E*>(a.k_cache) + base;
  const E* vp = reinterpret_cast<const E*>(a.v_cache) + base;
#pragma unroll
  for (int r = 0; r < D / (4 * X); ++r) f.k[r] = T::load_chunk(kp + ((4 * r + grp) * kBlock + n) * X);
#pragma unroll
  for (int mt = 0; mt < D / 16; ++mt) f.v[mt] = T::load_v(vp + (16 * mt + n) * kBlock + 4 * grp);
}

// Scores -> probabilities -> PV for one 16-key block.  Scores are scaled to
// log2 units first (s2 = s * scale * log2(e)).  The softmax keeps a lazily
// moved reference maximum m per row: probabilities are 2^(s2 - m), and m
// (with the O / l rescale it implies) only moves when some score of the wave
// exceeds it by more than 8, so probabilities stay <= 2^8 and the
// accumulators are rescaled on a few blocks only.  The quotient O / l at the
// end is the same for any m; the block that sets m has its maximum at
// exactly 2^0 = 1, so a single key returns its value row unchanged.
// `edge` (wave-uniform) marks a block with keys past kend or past some row's
// causal limit; only then are scores masked and V rows of keys >= kend zeroed.
template <int DT, int D>
__device__ inline void consume_block(const AttnArgs& a, const typename Tr<DT>::Chunk* qf, const BlockFrags<DT, D>& f,
                                     int kb, int kend, int limit, bool edge, bool few_keys, RowState<DT, D>& st) {
  using T = Tr<DT>;
  constexpr int R = D / (4 * T::X);
  constexpr int MT = D / 16;
  const int grp = (threadIdx.x & 63) >> 4;
  f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int r = 0; r < R; ++r) s = T::qk(f.k[r], qf[r], s);
  s *= a.scale_log2;
  const int key0 = kb * kBlock + 4 * grp;
  if (edge) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (!(key0 + i <= limit && key0 + i < kend)) s[i] = -INFINITY;
  }
  const float lmax = fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3]));
  if (__any(lmax > st.m + 8.f)) {
    float bm = fmaxf(lmax, __shfl_xor(lmax, 16));
    bm = fmaxf(bm, __shfl_xor(bm, 32));
    const float m_new = fmaxf(st.m, bm);
    const float alpha = m_new == -INFINITY ? 1.f : exp2_fast(st.m - m_new);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) st.acc[mt] *= alpha;
    st.l *= alpha;
    st.m = m_new;
  }
  // rows whose reference is still -inf have seen no visible key: p = 0
  const float m = st.m == -INFINITY ? 0.f : st.m;
  f32x4 p;
#pragma unroll
  for (int i = 0; i < 4; ++i) p[i] = exp2_fast(s[i] - m);
  const auto pf = T::make_p(p);
  st.l = T::psum(p, pf, st.l);
  if constexpr (T::kRoundsP) {
    if (few_keys) {
      // rows of at most kFewKeys keys: few probabilities carry each output,
      // so their bf16 rounding would not average out; the remainder p - hi
      // goes through a second PV product
      const auto plo = T::make_p_lo(p, pf);
      st.l = T::psum(p, plo, st.l);
      const int nvalid = edge ? kend - key0 : kBlock;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const auto v = T::keep_first(f.v[mt], nvalid);
        st.acc[mt] = T::pv(v, plo, T::pv(v, pf, st.acc[mt]));
      }
      return;
    }
  }
  if (edge) {
    const int nvalid = kend - key0;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) st.acc[mt] = T::pv(T::keep_first(f.v[mt], nvalid), pf, st.acc[mt]);
  } else {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) st.acc[mt] = T::pv(f.v[mt], pf, st.acc[mt]);
  }
}

// Blocks kb_begin .. kb_end-1 for 16 rows whose smallest causal limit is
// min_limit.  Software-pipelined one block deep: the next block's fragments
// are requested before the current one is consumed (the request is pinned in
// place with a scheduling barrier, and is issued unconditionally -- the last
// block is requested twice -- so consuming a block waits only for its own
// loads).  One block deep keeps the decode kernel at 3 waves per SIMD; two
// deep costs a wave per SIMD and measured slower.  Block ids come from a
// coalesced load of up to 64 consecutive block-table entries, one per lane,
// broadcast with readlane.
template <int DT, int D>
__device__ inline void attend_blocks(const AttnArgs& a, const typename Tr<DT>::Chunk* qf,
                                     const int32_t* bt, int g, int kb_begin, int kb_end, int kend,
                                     int limit, int min_limit, RowState<DT, D>& st, bool& poison) {
  const int lane = threadIdx.x & 63;
  const bool few_keys = kend <= kFewKeys;  // every row sees at most kFewKeys keys
  for (int c0 = kb_begin; c0 < kb_end; c0 += 64) {
    const int c1 = min(kb_end, c0 + 64);
    const int ids = c0 + lane < c1 ? bt[c0 + lane] : 0;
    auto block_id = [&](int kb) -> int {
      int blk = __builtin_amdgcn_readlane(ids, min(kb, c1 - 1) - c0);
      if (blk < 0 || blk >= a.nb) {
        poison = true;
        blk = 0;
      }
      return blk;
    };
    auto is_edge = [&](int kb) { return kb * kBlock + kBlock > kend || kb * kBlock + kBlock - 1 > min_limit; };
    BlockFrags<DT, D> fa, fb;
    load_block<DT, D>(a, block_id(c0), g, fa);
    for (int kb = c0; kb < c1; kb += 2) {
      load_block<DT, D>(a, block_id(kb + 1), g, fb);
      __builtin_amdgcn_sched_barrier(0);
      consume_block<DT, D>(a, qf, fa, kb, kend, limit, is_edge(kb), few_keys, st);
      if (kb + 1 >= c1) break;
      load_block<DT, D>(a, block_id(kb + 2), g, fa);
      __builtin_amdgcn_sched_barrier(0);
      consume_block<DT, D>(a, qf, fb, kb + 1, kend, limit, is_edge(kb + 1), few_keys, st);
    }
  }
}

// attend_blocks for fp8 caches.  A block's K and V granules of one head are
// 16 * D bytes each; read into registers in the MFMA operand layout they take
// 8-byte (K) and 4-byte (V) loads per lane, and such narrow loads stream
// about a tenth slower than 16-byte ones from scattered granules.  So each
// wave copies whole granules into a private ring of three LDS slots with
// 16-byte direct-to-LDS loads (non-temporal, 1 KB per instruction), two
// blocks ahead of the one it consumes, and reads the codes from LDS in the
// operand layout (conflict-free: a wave's K read covers 512 contiguous
// bytes, its V read 256).  `ring` is the wave's 3 * 2 * 16 * D bytes of LDS.
// The copies are counted in vmcnt only (the compiler does not see them), so
// the waits are explicit; the loop issues no other vector-memory operation.
template <int D>
__device__ inline void attend_blocks_fp8_lds(const AttnArgs& a, const bf16x8* qf, const int32_t* bt, int g,
                                             int kb_begin, int kb_end, int kend, int limit, int min_limit,
                                             RowState<2, D>& st, bool& poison, uint8_t* ring) {
  using T = Tr<2>;
  constexpr int GB = kBlock * D;    // bytes of one granule (K or V of one block and head)
  constexpr int NI = GB / 1024;     // 1 KB copies per granule
  constexpr int SLOT = 2 * GB;      // K granule, then V granule
  constexpr int R = D / (4 * T::X);
  constexpr int MT = D / 16;
  static_assert(GB % 1024 == 0, "whole 1 KB copies");
  const int lane = threadIdx.x & 63;
  const int n = lane & 15, grp = lane >> 4;
  const bool few_keys = kend <= kFewKeys;
  for (int c0 = kb_begin; c0 < kb_end; c0 += 64) {
    const int c1 = min(kb_end, c0 + 64);
    const int ids = c0 + lane < c1 ? bt[c0 + lane] : 0;
    auto block_id = [&](int kb) -> int {
      int blk = __builtin_amdgcn_readlane(ids, min(kb, c1 - 1) - c0);
      if (blk < 0 || blk >= a.nb) {
        poison = true;
        blk = 0;
      }
      return blk;
    };
    auto copy = [&](int kb, int slot) {
      const size_t gran = ((size_t)block_id(kb) * a.hkv + g) * GB;
      const uint8_t* kp = reinterpret_cast<const uint8_t*>(a.k_cache) + gran;
      const uint8_t* vp = reinterpret_cast<const uint8_t*>(a.v_cache) + gran;
#pragma unroll
      for (int u = 0; u < NI; ++u) {
        global_to_lds16_nt(kp, (unsigned)(u * 1024 + lane * 16), ring + slot * SLOT + u * 1024);
        global_to_lds16_nt(vp, (unsigned)(u * 1024 + lane * 16), ring + slot * SLOT + GB + u * 1024);
      }
    };
    copy(c0, 0);
    copy(c0 + 1, 1);  // past the chunk's last block: that block again (unused)
    int slot = 0;
    for (int kb = c0; kb < c1; ++kb) {
      copy(kb + 2, slot == 0 ? 2 : slot - 1);
      MPA_WAIT_VMCNT(4 * NI);  // the copies of blocks kb+1 and kb+2 may still be in flight
      const uint8_t* sp = ring + slot * SLOT;
      BlockFrags<2, D> f;
#pragma unroll
      for (int r = 0; r < R; ++r)
        f.k[r] = T::k_from_codes(*reinterpret_cast<const u32x2*>(sp + ((4 * r + grp) * kBlock + n) * T::X));
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        f.v[mt] = T::v_from_codes(*reinterpret_cast<const unsigned*>(sp + GB + (16 * mt + n) * kBlock + 4 * grp));
      const bool edge = kb * kBlock + kBlock > kend || kb * kBlock + kBlock - 1 > min_limit;
      consume_block<2, D>(a, qf, f, kb, kend, limit, edge, few_keys, st);
      slot = slot == 2 ? 0 : slot + 1;
    }
    // The ring is reused by the next group of blocks (and the wave's LDS is
    // released when it ends): no copy may still be writing it.
    MPA_WAIT_VMCNT(0);
  }
}

template <int D>
__device__ inline void store_fp8_chunk(const AppendArgs& a, size_t head, int c, int slot, u32x4 kw, u32x4 vw);

// A decode row's new token (query row t, position pos) for KV head g,
// written by the wave that reads the row's last split -- split edges are
// block-aligned, so no other wave reads this (block, head) granule -- with
// the bits the append kernels store (E4M3 codes for fp8 caches).  The wave
// then waits for its stores before it loads any block.  A bad block id
// writes nothing (the row comes out NaN).
template <int DT, int D>
__device__ inline void append_decode_token(const AttnArgs& a, int s, int pos, int t, int g) {
  using T = Tr<DT>;
  using E = typename T::Elem;
  constexpr int X = T::X;
  const int lane = threadIdx.x & 63;
  const int blk = a.block_tables[(size_t)s * a.mb + pos / kBlock];
  if (blk < 0 || blk >= a.nb) return;
  const int slot = pos % kBlock;
  const size_t head = (size_t)blk * a.hkv + g;
  if constexpr (DT == 2) {
    AppendArgs aa;
    aa.k_cache = const_cast<void*>(a.k_cache);
    aa.v_cache = const_cast<void*>(a.v_cache);
    aa.inv_k_scale = a.inv_k_scale;
    aa.inv_v_scale = a.inv_v_scale;
    const uint16_t* kn = reinterpret_cast<const uint16_t*>(a.k_new) + ((size_t)t * a.hkv + g) * D;
    const uint16_t* vn = reinterpret_cast<const uint16_t*>(a.v_new) + ((size_t)t * a.hkv + g) * D;
    for (int c = lane; c < D / 8; c += 64)
      store_fp8_chunk<D>(aa, head, c, slot, *reinterpret_cast<const u32x4*>(kn + c * 8),
                         *reinterpret_cast<const u32x4*>(vn + c * 8));
  } else {
    constexpr int NC = D / X;
    const size_t src = ((size_t)t * a.hkv + g) * D;
    for (int c = lane; c < NC; c += 64) {
      const u32x4 kv = *reinterpret_cast<const u32x4*>(reinterpret_cast<const E*>(a.k_new) + src + c * X);
      E vv[X];
#pragma unroll
      for (int e = 0; e < X; ++e) vv[e] = reinterpret_cast<const E*>(a.v_new)[src + c * X + e];
      *reinterpret_cast<u32x4*>(reinterpret_cast<E*>(const_cast<void*>(a.k_cache)) +
                                ((head * NC + c) * kBlock + slot) * X) = kv;
      E* vc = reinterpret_cast<E*>(const_cast<void*>(a.v_cache)) + (head * D + c * X) * kBlock + slot;
#pragma unroll
      for (int e = 0; e < X; ++e) vc[e * kBlock] = vv[e];
    }
  }
  MPA_WAIT_VMCNT(0);  // stores are counted in vmcnt: complete before the first block load
}

// ---------------------------------------------------------------------------
// Decode: one wave per (sequence, split, KV head); the G query heads of the
// group are the 16 MFMA columns (columns >= G carry zero queries).
template <int DT, int D>
__global__ __launch_bounds__(256) void decode_kernel(AttnArgs a, DecodePlan p) {
  using T = Tr<DT>;
  using QE = typename T::QElem;
  constexpr int X = T::X;
  constexpr int R = D / (4 * X);
  constexpr int MT = D / 16;
  const int lane = threadIdx.x & 63;
  const int wave = wave_uniform(threadIdx.x >> 6);
  const int unit = blockIdx.x * kWavesPerGroup + wave;
  const int item = unit / a.hkv;
  if (item >= p.item_start[p.n_seqs]) return;
  const int g = unit - item * a.hkv;
  const int j = upper_index(p.item_start, p.n_seqs, item);
  const int s = p.seq[j];
  const int split = item - p.item_start[j];
  const int nsplit = p.item_start[j + 1] - p.item_start[j];
  const int L = a.seq_lens[s];
  const int k0 = split * p.split_tokens[j];
  const int k1 = min(L, k0 + p.split_tokens[j]);
  const int trow = a.qsl[s];
  const int G = a.hq / a.hkv;
  const int n = lane & 15, grp = lane >> 4;
  const bool head_ok = n < G;
  const int h = g * G + (head_ok ? n : 0);
  if (a.k_new != nullptr && split == nsplit - 1) append_decode_token<DT, D>(a, s, L - 1, trow, g);

  const QE* q = reinterpret_cast<const QE*>(a.q) + ((size_t)trow * a.hq + h) * D;
  typename T::Chunk qf[R];
#pragma unroll
  for (int r = 0; r < R; ++r) qf[r] = head_ok ? T::load_q(q + (4 * r + grp) * X) : T::zero_chunk();

  RowState<DT, D> st;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) st.acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  st.m = -INFINITY;
  st.l = 0.f;
  bool poison = false;
  if constexpr (DT == 2) {
    __shared__ __attribute__((aligned(16))) uint8_t ring[kWavesPerGroup][3 * 2 * kBlock * D];
    attend_blocks_fp8_lds<D>(a, qf, a.block_tables + (size_t)s * a.mb, g, k0 / kBlock, (k1 + kBlock - 1) / kBlock,
                             k1, INT32_MAX, INT32_MAX, st, poison, ring[wave]);
  } else {
    attend_blocks<DT, D>(a, qf, a.block_tables + (size_t)s * a.mb, g, k0 / kBlock, (k1 + kBlock - 1) / kBlock, k1,
                         INT32_MAX, INT32_MAX, st, poison);
  }

  float l = st.l + __shfl_xor(st.l, 16);
  l += __shfl_xor(l, 32);
  if (!head_ok) return;
  if (nsplit == 1) {
    const float inv = poison ? NAN : a.v_scale / l;
    QE* o = reinterpret_cast<QE*>(a.out) + ((size_t)trow * a.hq + h) * D;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) T::store4(o + 16 * mt + 4 * grp, st.acc[mt] * inv);
    if (a.lse && grp == 0) a.lse[(size_t)trow * a.hq + h] = poison ? NAN : (st.m + log2f(l)) * kLn2;
  } else {
    const size_t slot = (size_t)(p.item_base + item) * a.hq + h;
    float* wo = a.ws_o + slot * D;
    const float bad = poison ? NAN : 1.f;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
      *reinterpret_cast<f32x4*>(wo + 16 * mt + 4 * grp) = st.acc[mt] * (bad * a.v_scale);
    if (grp == 0) {
      a.ws_ml[slot * 2] = st.m;
      a.ws_ml[slot * 2 + 1] = l * bad;
    }
  }
}

// Split-K merge.  With split maxima m_k and sums l_k (log2 units), a row's
// softmax denominator is sum_k l_k 2^(m_k - M) with M = max_k m_k, and its
// output is sum_k acc_k 2^(m_k - M) divided by that denominator.
//
// One output row from n partial results, by one wave.  Splits are taken 64
// at a time: lane k loads split k's (m, l) pair, the group's maximum and
// weighted sum come from wave reductions, and the partial rows are then
// loaded four at a time (all four issued before any is used), each weight
// broadcast from its lane.  Only the n real splits are read.  ml points at
// split 0's (m, l) pair (8-byte aligned), acc at split 0's element `lane` of
// the row; consecutive splits are ml_stride and acc_stride floats apart.
// Lane l writes elements l, l + 64, ... of out; lane 0 writes lse.
__device__ inline float wave_max64(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x = fmaxf(x, __shfl_xor(x, off));
  return x;
}
__device__ inline float wave_sum64(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
  return x;
}
__device__ inline float lane_value(float x, int k) {  // k wave-uniform
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), k));
}

template <int DT, int D>
__device__ inline void merge_splits(const float* ml, size_t ml_stride, const float* acc, size_t acc_stride, int n,
                                    typename Tr<DT>::QElem* out, float* lse) {
  using T = Tr<DT>;
  constexpr int PER = D / 64;
  constexpr int U = 4;
  const int lane = threadIdx.x & 63;
  float M = -INFINITY, lsum = 0.f;
  float o[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) o[e] = 0.f;
  for (int c0 = 0; c0 < n; c0 += 64) {
    const int cnt = min(64, n - c0);
    float mk = -INFINITY, lk = 0.f;
    if (lane < cnt) {
      const float2 v = *reinterpret_cast<const float2*>(ml + (size_t)(c0 + lane) * ml_stride);
      mk = v.x;
      lk = v.y;
    }
    const float gm = fmaxf(M, wave_max64(mk));      // every split holds a key: finite
    const float wk = lane < cnt ? exp2_fast(mk - gm) : 0.f;
    const float rescale = exp2_fast(M - gm);        // M = -inf on the first group: 0
    lsum = lsum * rescale + wave_sum64(wk * lk);
#pragma unroll
    for (int e = 0; e < PER; ++e) o[e] *= rescale;
    const float* a0 = acc + (size_t)c0 * acc_stride;
    int k = 0;
    for (; k + U <= cnt; k += U) {
      float v[U][PER];
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < PER; ++e) v[u][e] = a0[(size_t)(k + u) * acc_stride + 64 * e];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float w = lane_value(wk, k + u);
#pragma unroll
        for (int e = 0; e < PER; ++e) o[e] += w * v[u][e];
      }
    }
    for (; k < cnt; ++k) {
      const float w = lane_value(wk, k);
#pragma unroll
      for (int e = 0; e < PER; ++e) o[e] += w * a0[(size_t)k * acc_stride + 64 * e];
    }
    M = gm;
  }
  const float inv = 1.f / lsum;
#pragma unroll
  for (int e = 0; e < PER; ++e) T::store1(out + lane + 64 * e, o[e] * inv);
  if (lse && lane == 0) *lse = (M + log2f(lsum)) * kLn2;
}

// The merge kernels run four waves per workgroup, each wave merging whole
// (row, q head) pairs on its own (no LDS, no barrier): a launch with one
// small workgroup per pair is bound by the dispatcher's workgroup rate
// (about 1.2 per ns), not by the bytes it moves.
constexpr int kMergeWaves = 4;
constexpr int kPrefillMergeHeadsPerWave = 4;

// Decode merge: one workgroup per (split decode sequence, 4 q heads); wave w
// merges head 4 * blockIdx.y + w.
template <int DT, int D>
__global__ __launch_bounds__(64 * kMergeWaves) void merge_kernel(AttnArgs a, DecodePlan p) {
  using E = typename Tr<DT>::QElem;
  const int j = blockIdx.x;
  const int h = blockIdx.y * kMergeWaves + wave_uniform(threadIdx.x >> 6);
  if (j >= p.n_seqs || h >= a.hq) return;
  const int n = p.item_start[j + 1] - p.item_start[j];
  if (n <= 1) return;
  const int s = p.seq[j];
  const size_t base = (size_t)p.item_base + p.item_start[j];
  const int t = a.qsl[s];
  const int lane = threadIdx.x & 63;
  merge_splits<DT, D>(a.ws_ml + (base * a.hq + h) * 2, (size_t)a.hq * 2,
                      a.ws_o + (base * a.hq + h) * D + lane, (size_t)a.hq * D, n,
                      reinterpret_cast<E*>(a.out) + ((size_t)t * a.hq + h) * D,
                      a.lse ? a.lse + (size_t)t * a.hq + h : nullptr);
}

// Prefill merge: one workgroup per (token of a KV-split chunk, 16 q heads);
// wave w merges heads 16 * blockIdx.y + w + 4 * k, k < 4.  Split x of token
// i of chunk j sits at slot item_base[j] + x*C + i.
template <int DT, int D>
__global__ __launch_bounds__(64 * kMergeWaves) void prefill_merge_kernel(AttnArgs a, PrefillPlan p) {
  using E = typename Tr<DT>::QElem;
  const int r = blockIdx.x;
  if (r >= p.row_start[p.n_seqs]) return;
  const int j = upper_index(p.row_start, p.n_seqs, r);
  const int s = p.seq[j];
  const int i = r - p.row_start[j];
  const int t0 = a.qsl[s];
  const int C = a.qsl[s + 1] - t0;
  const size_t slot = (size_t)p.item_base[j] + i;
  const int lane = threadIdx.x & 63;
  const int h0 = blockIdx.y * (kMergeWaves * kPrefillMergeHeadsPerWave) + wave_uniform(threadIdx.x >> 6);
  for (int k = 0; k < kPrefillMergeHeadsPerWave; ++k) {
    const int h = h0 + k * kMergeWaves;
    if (h >= a.hq) break;
    merge_splits<DT, D>(a.ws_ml + (slot * a.hq + h) * 2, (size_t)C * a.hq * 2,
                        a.ws_o + (slot * a.hq + h) * D + lane, (size_t)C * a.hq * D, p.nsplit[j],
                        reinterpret_cast<E*>(a.out) + ((size_t)(t0 + i) * a.hq + h) * D,
                        a.lse ? a.lse + (size_t)(t0 + i) * a.hq + h : nullptr);
  }
}

// ---------------------------------------------------------------------------
// Prefill chunks: one workgroup per (sequence, query tile, KV head).  The
// tile's 64 (token, head) rows are the 16 columns of each of the 4 waves;
// row r is token r / G of the tile and head r % G of the group.
template <int DT, int D>
__global__ __launch_bounds__(256) void prefill_kernel(AttnArgs a, PrefillPlan p) {
  using T = Tr<DT>;
  using QE = typename T::QElem;
  constexpr int X = T::X;
  constexpr int R = D / (4 * X);
  constexpr int MT = D / 16;
  const int lane = threadIdx.x & 63;
  const int wave = wave_uniform(threadIdx.x >> 6);
  const int tile = blockIdx.x;
  const int g = blockIdx.y;
  if (tile >= p.tile_start[p.n_seqs]) return;
  const int j = upper_index(p.tile_start, p.n_seqs, tile);
  const int s = p.seq[j];
  const int qt = tile - p.tile_start[j];
  const int t0 = a.qsl[s];
  const int C = a.qsl[s + 1] - t0;
  const int L = a.seq_lens[s];
  const int P = L - C;
  const int G = a.hq / a.hkv;
  const int first_tok = qt * p.q_tile;
  if (first_tok + (wave * 16) / G >= C) return;  // this wave has no rows
  const int n = lane & 15, grp = lane >> 4;
  const int row = wave * 16 + n;
  // The tile holds q_tile tokens (G * q_tile <= 64 rows): when G does not
  // divide 64, the last rows of the workgroup would fall on the next tile's
  // first token.  They compute a valid token of this tile and store nothing.
  const int r_tok = row / G;
  const int i_raw = first_tok + min(r_tok, p.q_tile - 1);
  const bool row_ok = r_tok < p.q_tile && i_raw < C;
  const int i = min(i_raw, C - 1);
  const int h = g * G + row % G;
  const int last_tok = min(first_tok + min((wave * 16 + 15) / G, p.q_tile - 1), C - 1);
  const int kend = P + last_tok + 1;  // keys this wave needs

  const QE* q = reinterpret_cast<const QE*>(a.q) + ((size_t)(t0 + i) * a.hq + h) * D;
  typename T::Chunk qf[R];
#pragma unroll
  for (int r = 0; r < R; ++r) qf[r] = T::load_q(q + (4 * r + grp) * X);

  RowState<DT, D> st;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) st.acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  st.m = -INFINITY;
  st.l = 0.f;
  bool poison = false;
  const int min_limit = P + min(first_tok + (wave * 16) / G, C - 1);
  attend_blocks<DT, D>(a, qf, a.block_tables + (size_t)s * a.mb, g, 0, (kend + kBlock - 1) / kBlock,
                       kend, P + i, min_limit, st, poison);

  float l = st.l + __shfl_xor(st.l, 16);
  l += __shfl_xor(l, 32);
  if (!row_ok) return;
  const float inv = poison ? NAN : a.v_scale / l;
  QE* o = reinterpret_cast<QE*>(a.out) + ((size_t)(t0 + i) * a.hq + h) * D;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) T::store4(o + 16 * mt + 4 * grp, st.acc[mt] * inv);
  if (a.lse && grp == 0)
    a.lse[(size_t)(t0 + i) * a.hq + h] = poison ? NAN : (st.m + log2f(l)) * kLn2;
}

// ---------------------------------------------------------------------------
// Prefill chunks, bf16: the tensor-core path.  One workgroup of WAVES waves
// per (sequence, 32*WAVES-row query tile, KV head); row r of the tile is token
// r / G and head r % G of the group, so the G heads that share a KV head share
// every K/V tile.  Each wave owns 32 rows (one 32-wide MFMA column tile).
//
// Per 64-key tile (4 cache blocks), in a STAGES-deep LDS ring:
//   S^T[64 keys][32 rows] = K . Q^T   2 x (D/16) v_mfma_f32_32x32x16_bf16
//   O^T[D][32 rows]     += V^T . P^T  (D/32) x 4 v_mfma_f32_32x32x16_bf16
// Tiles are fetched straight into LDS (global_load_lds, 16 bytes a lane) by
// the waves themselves, STAGES-1 tiles ahead of use, so no registers stage
// them and a copy has STAGES-1 tiles of compute to land in.  The per-lane
// source addresses permute 16-byte pieces so that every MFMA operand read
// from LDS is one contiguous run per 16 lanes (no bank conflicts):
//  * row m of a 32-key S^T tile is key 16(m/16) + swap23(m%16), where swap23
//    exchanges bits 2 and 3.  Then the 8 keys a lane holds for one 16-key PV
//    step (output rows 8j+4h+i, j in {2t', 2t'+1}) are keys 8h..8h+7 of the
//    block.  LDS holds each K chunk row with its 16 slots already in that
//    order: [block][d/8 chunks][slot][8], slot s = key swap23(s);
//  * LDS holds V^T as [block][key half h][d][8 keys], so lane (m, h) of a PV
//    step reads row 32dt+m of half h.
// Each wave copies a contiguous part of one block of a tile, so it needs one
// block id per tile (a scalar load) and fixes up its own pieces (zeroing V entries of keys >= L,
// which may hold NaN/Inf; NaN for an invalid block id) before the barrier
// that publishes the tile.
//
// Softmax: exact online softmax with a lazily updated reference maximum.  The
// running reference m only moves when a row's new maximum exceeds it by more
// than 8 (log2 units), so exp2(s - m) <= 2^8 and the O / l rescale is skipped
// for almost every tile; the final O / l is the same quotient either way.
template <int CT, int D, int WAVES, int STAGES>
__global__ __launch_bounds__(64 * WAVES, 1) void prefill_mfma_kernel(AttnArgs a, PrefillPlan p) {
  using f32x16 = float __attribute__((ext_vector_type(16)));
  using cint = const __attribute__((address_space(4))) int32_t;
  constexpr int BN = 64;                   // keys per tile
  constexpr int NB = BN / kBlock;          // cache blocks per tile
  constexpr int BLK = kBlock * D;          // elements of one (block, head) granule
  constexpr int TILE = NB * BLK;           // elements of one K (or V) tile
  constexpr int KS = D / 16;               // k-steps of the QK^T product
  static_assert(KS >= 4, "the V reads follow the last four k-steps");
  constexpr int DT = D / 32;               // 32-dim row tiles of O^T
  constexpr int NI = TILE * 2 / 1024;      // 1 KB copies per tile and cache
  constexpr int WI = NI / WAVES;           // ... per wave
  static_assert(WI >= 1 && NI % WAVES == 0 && (WI * 512) <= BLK && BLK % (WI * 512) == 0,
                "each wave copies part of exactly one block per tile");
  // CT: the cache type, 0 bf16 or 2 fp8.  fp8 codes take a register path:
  // each lane loads one 16-byte piece of the K tile and one of the V tile
  // (a (block, head) granule has D such pieces), one tile ahead, and at the
  // end of the iteration converts them to bf16 into the same LDS layout the
  // bf16 copies fill, so the compute below is the same for both.
  static_assert(CT == 0 || CT == 2, "bf16 or fp8 caches");
  static_assert(CT == 0 || (NB * D <= 64 * WAVES && (64 * WAVES) % D == 0), "one fp8 piece per lane");
  constexpr int AHEAD = CT == 2 ? 1 : STAGES - 1;  // tiles a copy runs ahead of its use
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  uint16_t* const sk = smem;                   // STAGES K tiles
  uint16_t* const sv = smem + STAGES * TILE;   // STAGES V tiles

  const int lane = threadIdx.x & 63;
  const int wave = wave_uniform(threadIdx.x >> 6);
  const int n_tiles = p.tile_start[p.n_seqs];
  const int g = blockIdx.x % a.hkv;
  const int tile = n_tiles - 1 - (int)(blockIdx.x / a.hkv);  // last (longest) query tiles first
  const int j = upper_index(p.tile_start, p.n_seqs, tile);
  const int s = p.seq[j];
  const int nsplit = p.nsplit[j];
  const int qt = (tile - p.tile_start[j]) / nsplit;
  const int split = tile - p.tile_start[j] - qt * nsplit;
  const int t0 = a.qsl[s];
  const int C = a.qsl[s + 1] - t0;
  const int L = a.seq_lens[s];
  const int P = L - C;
  const int G = a.hq / a.hkv;
  const int first_tok = qt * p.q_tile;
  const int last_tok = min(first_tok + p.q_tile - 1, C - 1);
  const int kend = P + last_tok + 1;  // keys the query tile needs
  // this workgroup's 64-key tiles: [kt_begin, ntile)
  const int kt_begin = split * p.split_tiles[j];
  const int ntile = split == nsplit - 1 ? (kend + BN - 1) / BN : kt_begin + p.split_tiles[j];
  cint* bt = (cint*)(a.block_tables + (size_t)s * a.mb);

  // this lane's query row.  The tile holds q_tile tokens (G * q_tile <= 256
  // rows): when G does not divide 256, the last rows of the workgroup would
  // fall on the next tile's first token, past the keys loaded here.  They
  // compute a valid token of this tile and store nothing.
  const int n = lane & 31, h = lane >> 5;
  const int row = wave * 32 + n;
  const int r_tok = row / G;
  const int i_raw = first_tok + min(r_tok, p.q_tile - 1);
  const bool row_ok = r_tok < p.q_tile && i_raw < C;
  const int i = min(i_raw, C - 1);
  const int head = g * G + row % G;
  const int limit = P + i;
  const int w_first = first_tok + (wave * 32) / G;
  const bool wave_active = w_first < C;
  const int w_min_limit = P + min(w_first, C - 1);
  const int w_kend = P + min(first_tok + min((wave * 32 + 31) / G, p.q_tile - 1), C - 1) + 1;

  bf16x8 qf[KS];
  {
    const uint16_t* q = reinterpret_cast<const uint16_t*>(a.q) + ((size_t)(t0 + i) * a.hq + head) * D;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(q + (2 * ks + h) * 8));
  }

  // ---- global -> LDS tile copies (this wave's slices)
  const int nblk = (kend + kBlock - 1) / kBlock;
  const int pi = wave * 64 + lane;  // fp8: this lane's 16-byte piece of the tile
  const int my_bi = CT == 2 ? (wave * 64) / D : (wave * WI * 512) / BLK;  // the tile block this wave copies
  u32x4 kraw = {0u, 0u, 0u, 0u}, vraw = {0u, 0u, 0u, 0u};  // fp8 pieces in flight
  // Tile kt's copy.  A block index past the sequence's last needed block is
  // clamped to it (its keys are all masked and its V entries zeroed), so
  // every copy is issued, always 2*WI instructions per wave per tile.
  // the id of the block this wave copies for tile kt (a scalar load)
  auto tile_block = [&](int kt) -> int { return bt[min(kt * NB + my_bi, nblk - 1)]; };
  // Byte offsets of the bf16 granules: consecutive cache blocks are
  // blk_bytes apart, this KV head's granule head_bytes into its block (both
  // below 2^32 for any head count the shape check admits).
  const unsigned blk_bytes = (unsigned)a.hkv * (unsigned)(BLK * 2);
  const unsigned head_bytes = (unsigned)g * (unsigned)(BLK * 2);
  // which: 1 the K slices, 2 the V slices, 3 both
  auto copy_tile = [&](int blk_raw, int stage, int which = 3) -> int {
    const unsigned blk = (unsigned)blk_raw < (unsigned)a.nb ? (unsigned)blk_raw : 0u;
    if constexpr (CT == 2) {
      if (pi < NB * D) {
        const size_t gran = ((size_t)blk * a.hkv + g) * (kBlock * D) + (size_t)(pi % D) * 16;
        if (which & 1) kraw = *reinterpret_cast<const u32x4*>(reinterpret_cast<const uint8_t*>(a.k_cache) + gran);
        if (which & 2) vraw = *reinterpret_cast<const u32x4*>(reinterpret_cast<const uint8_t*>(a.v_cache) + gran);
      }
      (void)stage;
      return blk_raw;
    }
    const uint64_t gran = (uint64_t)blk * blk_bytes + head_bytes;
    const uint8_t* kbase = reinterpret_cast<const uint8_t*>(a.k_cache) + gran;
    const uint8_t* vbase = reinterpret_cast<const uint8_t*>(a.v_cache) + gran;
#pragma unroll
    for (int u = 0; u < WI; ++u) {
      const int ii = wave * WI + u;                 // 1 KB slice of the tile
      const int cq = (ii * 64) % (BLK / 8) + lane;  // 16-byte piece within the block
      // K: piece (chunk c, slot) <- key swap23(slot) of chunk c
      const int kc = cq >> 4, ks16 = cq & 15;
      const int kkey = (ks16 & 3) | ((ks16 & 4) << 1) | ((ks16 & 8) >> 1);
      if (which & 1) global_to_lds16(kbase, (unsigned)((kc * 16 + kkey) * 16), sk + stage * TILE + ii * 512);
      // V: piece (half vh, row d) <- keys 8vh..8vh+7 of V^T row d
      const int vh = cq / D, vd = cq % D;
      if (which & 2) global_to_lds16(vbase, (unsigned)((vd * kBlock + vh * 8) * 2), sv + stage * TILE + ii * 512);
    }
    return blk_raw;
  };
  // After this wave's copy of tile kt has landed: zero its V entries of keys
  // >= L (the tail of the sequence's last block, and clamped blocks), or fill
  // them with NaN when the block id was invalid.
  // the first tile whose block copied by this wave holds keys >= L
  const int nfull = L / kBlock;
  const int kt_fix_from = nfull <= my_bi ? 0 : (nfull - my_bi + NB - 1) / NB;
  auto fix_tile = [&](int kt, int blk_raw, int stage) {
    const bool bad = (unsigned)blk_raw >= (unsigned)a.nb;
    if (kt < kt_fix_from && !bad) return;
    const int nvalid_blk = L - (kt * NB + my_bi) * kBlock;
#pragma unroll
    for (int u = 0; u < WI; ++u) {
      const int ii = wave * WI + u;
      const int cq = (ii * 64) % (BLK / 8) + lane;
      const int vh = cq / D;
      uint16_t* piece = sv + stage * TILE + ii * 512 + lane * 8;
      const int nvalid = nvalid_blk - 8 * vh;
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (bad || e >= nvalid) piece[e] = bad ? (uint16_t)0x7FC0 : (uint16_t)0;
    }
  };
  // fp8: once this lane's pieces of tile kt have landed, store them as bf16
  // in the tile's stage -- K piece q (keys 2j, 2j+1 of chunk c = q/8, j = q%8)
  // at the slots of those keys, V piece q (V^T row q, 16 keys) as its two key
  // halves -- with the V entries of keys >= L zeroed (NaN for a bad block id)
  auto store_fp8_tile = [&](int kt, int blk_raw, int stage) {
    if (pi >= NB * D) return;
    const int b = pi / D, q = pi % D;
    uint8_t* kdst = reinterpret_cast<uint8_t*>(sk + stage * TILE + b * BLK);
    uint8_t* vdst = reinterpret_cast<uint8_t*>(sv + stage * TILE + b * BLK);
    const int c = q >> 3, j = q & 7;
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      const int key = 2 * j + x;
      const int slot = (key & 3) | ((key & 4) << 1) | ((key & 8) >> 1);  // the slot that holds this key
      const u32x4 w = {Tr<2>::cvt2(kraw[2 * x], false), Tr<2>::cvt2(kraw[2 * x], true),
                       Tr<2>::cvt2(kraw[2 * x + 1], false), Tr<2>::cvt2(kraw[2 * x + 1], true)};
      *reinterpret_cast<u32x4*>(kdst + (c * 16 + slot) * 16) = w;
    }
    const int nvalid = L - (kt * NB + b) * kBlock;
    const bool bad = !(blk_raw >= 0 && blk_raw < a.nb);
#pragma unroll
    for (int vh = 0; vh < 2; ++vh) {
      u32x4 w = {Tr<2>::cvt2(vraw[2 * vh], false), Tr<2>::cvt2(vraw[2 * vh], true),
                 Tr<2>::cvt2(vraw[2 * vh + 1], false), Tr<2>::cvt2(vraw[2 * vh + 1], true)};
      if (bad || nvalid < 8 * vh + 8) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const unsigned keep = (unsigned)(!bad && 8 * vh + e < nvalid);
          const unsigned fill = bad ? 0x7FC0u : 0u;
          const unsigned sh = 16 * (e & 1);
          const unsigned cur = (w[e >> 1] >> sh) & 0xFFFFu;
          w[e >> 1] = (w[e >> 1] & ~(0xFFFFu << sh)) | ((keep ? cur : fill) << sh);
        }
      }
      *reinterpret_cast<u32x4*>(vdst + (vh * D + q) * 16) = w;
    }
  };

  f32x16 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[dt][r] = 0.f;
  const float c = a.scale_log2;
  const float thresh = 8.f / c;  // 8 in log2 units, in raw score units
  float m_ref = -INFINITY;       // reference maximum, raw score units
  float l = 0.f;
  // K operand row of this lane: slot n%16 of block n/16 of a 32-key tile
  const int koff = (n >> 4) * BLK + (n & 15) * 8;

  // the Q fragments (ordinary loads) land before any tile copy is issued, so
  // that no wait inside the loop is ever needed for them
  MPA_WAIT_VMCNT(0);
  // Stages rotate: tile kt sits in stage kt % STAGES, kept as counters that
  // step each iteration (s_use for tile kt, s_next for kt+1, s_copy for
  // kt+AHEAD).  The block ids of the tiles copied but not yet fixed up wait
  // in ids[]: ids[0] is tile kt+1's, ids[AHEAD-1] tile kt+AHEAD's.
  auto wrap = [](int x) { return x >= STAGES ? x - STAGES : x; };
  int s_use = kt_begin % STAGES;
  int ids[AHEAD];
  // prologue: the split's first AHEAD tiles in flight, its first published
#pragma unroll
  for (int k = 0; k < AHEAD; ++k) ids[k] = copy_tile(tile_block(kt_begin + k), wrap(s_use + k));
  // each iteration loads the block id the next one copies (see below)
  int next_blk = tile_block(kt_begin + AHEAD);
  if constexpr (CT == 2) {
    MPA_WAIT_VMCNT(0);
    store_fp8_tile(kt_begin, ids[0], s_use);
  } else {
    MPA_WAIT_VMCNT(2 * WI * (STAGES - 2));
    fix_tile(kt_begin, ids[0], s_use);
  }
#pragma unroll
  for (int k = 0; k + 1 < AHEAD; ++k) ids[k] = ids[k + 1];
  __syncthreads();

  // Waves w and w + WAVES/2 share a SIMD and run the same phases; the issue
  // arbiter favours the older one, so the upper half finishes each tile
  // last and the lower half waits for it at the barrier.  Raising the upper
  // half's priority shortens that critical path.
  if (wave >= WAVES / 2) __builtin_amdgcn_s_setprio(1);
  for (int kt = kt_begin; kt < ntile; ++kt) {
    // tile kt+STAGES-1 is copied into the stage tile kt-1 used (all waves are
    // past it): by an active wave between its QK products, so that the
    // copy instructions are issued while the matrix core is busy
    const int cblk = next_blk;
    ids[AHEAD - 1] = cblk;
    const int s_next = wrap(s_use + 1), s_copy = wrap(s_use + AHEAD);
    const int key_base = kt * BN;
    if (wave_active && key_base < w_kend) {
      const uint16_t* K = sk + s_use * TILE;
      const uint16_t* V = sv + s_use * TILE;
      // The K operands of the first KUP k-steps are read from LDS before the
      // first MFMA, and each later k-step's KUP steps ahead of its use, each
      // into registers of its own: the reads' latency overlaps instead of
      // separating every MFMA pair (left to itself the scheduler reuses one
      // register quad for them all), and the eight waves do not queue all
      // of the tile's K reads at the LDS at once when the tile is published.
      constexpr int KUP = 3;
      bf16x8 kf[2][KS];
      auto read_k = [&](int ks) {
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
          kf[rt][ks] =
              __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(K + 2 * rt * BLK + koff + (2 * ks + h) * 128));
      };
#pragma unroll
      for (int ks = 0; ks < KUP; ++ks) read_k(ks);
      __builtin_amdgcn_sched_barrier(0);
      f32x16 st[2];
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int r = 0; r < 16; ++r) st[rt][r] = 0.f;
      // V operands: the reads of cache block t of the tile are issued after
      // k-step KS-4+t of the QK product, into registers whose K operands
      // that step has consumed.  Spread over the last four k-steps, the
      // eight waves' V reads do not all reach the LDS at once when the
      // products end, and they land while the softmax runs.
      bf16x8 vf[4][DT];
      // the two 32-key row tiles are independent accumulation chains:
      // interleave them so back-to-back MFMAs never wait on each other
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
          st[rt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[rt][ks], qf[ks], st[rt], 0, 0, 0);
        if (ks + KUP < KS) {
          __builtin_amdgcn_sched_barrier(0);
          read_k(ks + KUP);
          __builtin_amdgcn_sched_barrier(0);
        }
        // the next tile copy: bf16 tiles as their K slices after the third
        // k-step and their V slices after k-step KS/2 (the same step at
        // D = 64); fp8 pieces both after the first, since they must land
        // in registers by the end of this tile
        constexpr int k_ks = CT == 0 ? 2 : 0;
        constexpr int v_ks = CT == 0 ? KS / 2 : 0;
        if (ks == k_ks || ks == v_ks) {
          __builtin_amdgcn_sched_barrier(0);
          copy_tile(cblk, s_copy, (ks == k_ks ? 1 : 0) | (ks == v_ks ? 2 : 0));
          __builtin_amdgcn_sched_barrier(0);
        }
        if (ks >= KS - 4) {
          const int t = ks - (KS - 4);
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int dt = 0; dt < DT; ++dt)
            vf[t][dt] = __builtin_bit_cast(
                bf16x8, *reinterpret_cast<const u32x4*>(V + t * BLK + (h * D + n) * 8 + 32 * dt * 8));
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      // the next copy's block id: a scalar load shares the LDS wait counter
      // and may complete out of order, so issued here, after the last LDS
      // read of the tile, it only turns the PV waits into full ones, by
      // which time the V reads have long landed
      next_blk = tile_block(kt + AHEAD + 1);
      if (key_base + BN - 1 > w_min_limit) {
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int jr = r >> 2;
            const int key = key_base + 32 * rt + 16 * (jr >> 1) + 8 * h + 4 * (jr & 1) + (r & 3);
            if (key > limit) st[rt][r] = -INFINITY;
          }
      }
      // The reference maximum m_ref moves only when some score of the wave
      // exceeds it by more than thresh (probabilities stay <= 2^8).  On a
      // wave's first tile it is still -inf and is taken from the tile's row
      // maximum; on later tiles the probabilities are formed with the current
      // reference first, and since a score past the threshold makes its
      // probability -- and so this lane's row-sum partial -- at least 2^8
      // after bf16 rounding, the tile's maximum is taken only when some
      // lane's partial reaches 2^8.  Then S is recomputed from the operands
      // still in LDS (the same products in the same order, so the same
      // values), the reference is moved if the threshold is passed, and the
      // probabilities are formed again.  Either way the probabilities, the
      // row sums and the reference are those of taking the maximum on every
      // tile.
      auto row_max = [&](const f32x16 (&s)[2]) -> float {
        float m4[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
          for (int r = 0; r < 16; ++r) m4[r & 3] = fmaxf(m4[r & 3], s[rt][r]);
        return max_across_halves(fmaxf(fmaxf(m4[0], m4[1]), fmaxf(m4[2], m4[3])));
      };
      auto move_reference = [&](float mx) {
        const float m_new = fmaxf(m_ref, mx);
        const float alpha = m_new == -INFINITY ? 1.f : exp2_fast((m_ref - m_new) * c);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[dt] *= alpha;
        l *= alpha;
        m_ref = m_new;
      };
      // P^T in bf16; the row sum adds the rounded values the PV product
      // uses (four independent partial sums, two probabilities per dot2).
      bf16x8 pb[4];
      float l4[4];
      auto make_p = [&](const f32x16 (&s)[2], float mc) {
#pragma unroll
        for (int k = 0; k < 4; ++k) l4[k] = 0.f;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
#pragma unroll
          for (int e = 0; e < 8; ++e) pb[t][e] = (__bf16)exp2_fast(fmaf(s[t >> 1][8 * (t & 1) + e], c, -mc));
          const u32x4 w = __builtin_bit_cast(u32x4, pb[t]);
#pragma unroll
          for (int k = 0; k < 4; ++k) l4[k] = add_bf16_pair(w[k], l4[k]);
        }
      };
      if (kt == kt_begin) {
        const float mx = row_max(st);
        if (__any(mx > m_ref + thresh)) move_reference(mx);
      }
      make_p(st, m_ref * c);
      if (kt != kt_begin && __any(!((l4[0] + l4[1]) + (l4[2] + l4[3]) < 256.f))) {
        asm volatile("" ::: "memory");
        f32x16 s2[2];
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
          for (int r = 0; r < 16; ++r) s2[rt][r] = 0.f;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
          for (int rt = 0; rt < 2; ++rt)
            s2[rt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf16x8,
                                   *reinterpret_cast<const u32x4*>(K + 2 * rt * BLK + koff + (2 * ks + h) * 128)),
                qf[ks], s2[rt], 0, 0, 0);
        if (key_base + BN - 1 > w_min_limit) {
#pragma unroll
          for (int rt = 0; rt < 2; ++rt)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const int jr = r >> 2;
              const int key = key_base + 32 * rt + 16 * (jr >> 1) + 8 * h + 4 * (jr & 1) + (r & 3);
              if (key > limit) s2[rt][r] = -INFINITY;
            }
        }
        const float mx = row_max(s2);
        if (__any(mx > m_ref + thresh)) {
          move_reference(mx);
          make_p(s2, m_ref * c);
        }
      }
      const float mc = m_ref * c;
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[t][dt], pb[t], o[dt], 0, 0, 0);
      l += (l4[0] + l4[1]) + (l4[2] + l4[3]);
      if (key_base == 0 && w_min_limit < kFewKeys) {
        // A row that sees at most kFewKeys keys has them all in tile 0, and
        // its output rests on so few probabilities that their bf16 rounding
        // does not average out.  For such waves the tile is passed a second
        // time with the remainder p - bf16(p): S is recomputed from the
        // operands still in LDS (the same products in the same order, so
        // the same values), and the remainder goes into the PV product and
        // the row sum, which carries P to about 16 bits.  The empty asm
        // keeps the compiler from holding the first pass's fragments live
        // across the tile for this rare branch.
        asm volatile("" ::: "memory");
        f32x16 s2[2];
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
          for (int r = 0; r < 16; ++r) s2[rt][r] = 0.f;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
          for (int rt = 0; rt < 2; ++rt)
            s2[rt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf16x8,
                                   *reinterpret_cast<const u32x4*>(K + 2 * rt * BLK + koff + (2 * ks + h) * 128)),
                qf[ks], s2[rt], 0, 0, 0);
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int jr = r >> 2;
            const int key = 32 * rt + 16 * (jr >> 1) + 8 * h + 4 * (jr & 1) + (r & 3);
            if (key > limit) s2[rt][r] = -INFINITY;
          }
        float r4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          bf16x8 plo;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float pe = exp2_fast(fmaf(s2[t >> 1][8 * (t & 1) + e], c, -mc));
            plo[e] = (__bf16)(pe - (float)(__bf16)pe);
          }
          const u32x4 w = __builtin_bit_cast(u32x4, plo);
#pragma unroll
          for (int k = 0; k < 4; ++k) r4[k] = add_bf16_pair(w[k], r4[k]);
#pragma unroll
          for (int dt = 0; dt < DT; ++dt)
            o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(V + t * BLK + (h * D + n) * 8 + 32 * dt * 8)),
                plo, o[dt], 0, 0, 0);
        }
        l += (r4[0] + r4[1]) + (r4[2] + r4[3]);
      }
    } else {
      copy_tile(cblk, s_copy);
      next_blk = tile_block(kt + AHEAD + 1);
      // The block id is a scalar load, which shares the LDS counter and may
      // return out of order.  Left pending on this path, it would reach the
      // active path's join as well, and every wait for the K operand reads
      // there would become a wait for all of them.
      MPA_WAIT_LGKMCNT(0);
    }
    if constexpr (CT == 2) {
      // this lane's pieces of tile kt+1 (the only loads in flight)
      MPA_WAIT_VMCNT(0);
      store_fp8_tile(kt + 1, ids[0], s_next);
    } else {
      // this wave's part of tile kt+1 has landed once only the copies issued
      // after it (tiles kt+2 .. kt+STAGES-1) remain in flight
      MPA_WAIT_VMCNT(2 * WI * (STAGES - 2));
      fix_tile(kt + 1, ids[0], s_next);
    }
#pragma unroll
    for (int k = 0; k + 1 < AHEAD; ++k) ids[k] = ids[k + 1];
    s_use = s_next;
    __syncthreads();
  }
  MPA_WAIT_VMCNT(0);  // drain the clamped copies past the end

  const float lt = l + __shfl_xor(l, 32);
  if (!wave_active || !row_ok) return;
  if (nsplit > 1) {  // partial result of this KV split, merged by prefill_merge_kernel
    const size_t slot = ((size_t)p.item_base[j] + (size_t)split * C + i) * a.hq + head;
    float* wo = a.ws_o + slot * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int jb = 0; jb < 4; ++jb) {
        const f32x4 v4 = {o[dt][4 * jb], o[dt][4 * jb + 1], o[dt][4 * jb + 2], o[dt][4 * jb + 3]};
        *reinterpret_cast<f32x4*>(wo + 32 * dt + 8 * jb + 4 * h) = v4 * a.v_scale;
      }
    if (h == 0) {
      a.ws_ml[slot * 2] = m_ref * c;
      a.ws_ml[slot * 2 + 1] = lt;
    }
    return;
  }
  const float inv = a.v_scale / lt;
  uint16_t* out = reinterpret_cast<uint16_t*>(a.out) + ((size_t)(t0 + i) * a.hq + head) * D;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int jb = 0; jb < 4; ++jb) {
      f32x4 v4 = {o[dt][4 * jb], o[dt][4 * jb + 1], o[dt][4 * jb + 2], o[dt][4 * jb + 3]};
      Tr<0>::store4(out + 32 * dt + 8 * jb + 4 * h, v4 * inv);
    }
  if (a.lse && h == 0) a.lse[(size_t)(t0 + i) * a.hq + head] = (m_ref * c + log2f(lt)) * kLn2;
}

// Stores chunk c (8 consecutive bf16 elements, packed) of a new key row and
// of a new value row into slot `slot` of cache head `head` of an fp8 cache:
// each element x becomes the E4M3 code of x * (1 / scale).
template <int D>
__device__ inline void store_fp8_chunk(const AppendArgs& a, size_t head, int c, int slot, u32x4 kw, u32x4 vw) {
  constexpr int NC = D / 8;
  float kx[8], vx[8];
  Tr<0>::unpack(kw, kx);
  Tr<0>::unpack(vw, vx);
  u32x2 kc = {0u, 0u};
#pragma unroll
  for (int e = 0; e < 8; ++e) kc[e / 4] |= f32_to_e4m3(kx[e] * a.inv_k_scale) << (8 * (e % 4));
  *reinterpret_cast<u32x2*>(reinterpret_cast<uint8_t*>(a.k_cache) + ((head * NC + c) * kBlock + slot) * 8) = kc;
  uint8_t* vc = reinterpret_cast<uint8_t*>(a.v_cache) + (head * D + c * 8) * kBlock + slot;
#pragma unroll
  for (int e = 0; e < 8; ++e) vc[e * kBlock] = (uint8_t)f32_to_e4m3(vx[e] * a.inv_v_scale);
}

// ---------------------------------------------------------------------------
// Append: one wave per new token.  The token's sequence comes from the
// kernel-argument plan (directly when every sequence of the plan adds one
// token, else by a scalar binary search), its block id from one scalar load;
// the wave then copies the token's Hkv*d key elements as 16-byte chunks and
// its value elements into the V^T rows of the slot, issuing the loads of up
// to 4 chunks per lane before their stores.
template <int DT, int D>
__global__ __launch_bounds__(256) void append_kernel(AppendArgs a, AppendPlan p) {
  using T = Tr<DT>;
  using E = typename T::Elem;
  constexpr int X = T::X;
  constexpr int NC = D / X;
  constexpr int U = 4;
  const int lane = threadIdx.x & 63;
  const int tok = blockIdx.x * kWavesPerGroup + wave_uniform(threadIdx.x >> 6);
  if (tok >= p.tok_start[p.n_seqs]) return;
  const int j = p.unit ? tok : upper_index(p.tok_start, p.n_seqs, tok);
  const int k = tok - p.tok_start[j];
  const int s = p.seq[j];
  const int t = p.row0[j] + k;
  const int pos = p.pos0[j] + k;
  const int blk = a.block_tables[(size_t)s * a.mb + pos / kBlock];
  if (blk < 0 || blk >= a.nb) return;
  const int slot = pos % kBlock;
  const int nchunk = a.hkv * NC;
  if constexpr (DT == 2) {
    // fp8 cache: each bf16 element of the new rows is stored as the E4M3
    // code of x * (1 / scale); a lane handles 8 consecutive elements
    const uint16_t* kn = reinterpret_cast<const uint16_t*>(a.k_new) + (size_t)t * a.hkv * D;
    const uint16_t* vn = reinterpret_cast<const uint16_t*>(a.v_new) + (size_t)t * a.hkv * D;
    for (int ci = lane; ci < nchunk; ci += 64) {
      const int h = ci / NC, c = ci - h * NC;
      store_fp8_chunk<D>(a, (size_t)blk * a.hkv + h, c, slot, *reinterpret_cast<const u32x4*>(kn + h * D + c * 8),
                         *reinterpret_cast<const u32x4*>(vn + h * D + c * 8));
    }
  } else {
  for (int c0 = 0; c0 < nchunk; c0 += 64 * U) {
    u32x4 kv[U];
    E vv[U][X];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int ci = min(c0 + 64 * u + lane, nchunk - 1);
      const int h = ci / NC, c = ci - h * NC;
      const size_t src = ((size_t)t * a.hkv + h) * D + c * X;
      kv[u] = *reinterpret_cast<const u32x4*>(reinterpret_cast<const E*>(a.k_new) + src);
#pragma unroll
      for (int e = 0; e < X; ++e) vv[u][e] = reinterpret_cast<const E*>(a.v_new)[src + e];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int ci = c0 + 64 * u + lane;
      if (ci >= nchunk) continue;
      const int h = ci / NC, c = ci - h * NC;
      const size_t head = (size_t)blk * a.hkv + h;
      *reinterpret_cast<u32x4*>(reinterpret_cast<E*>(a.k_cache) + ((head * NC + c) * kBlock + slot) * X) = kv[u];
      E* vc = reinterpret_cast<E*>(a.v_cache) + (head * D + c * X) * kBlock + slot;
#pragma unroll
      for (int e = 0; e < X; ++e) vc[e * kBlock] = vv[u][e];
    }
  }
  }
}

// Append for sequences that add several tokens: one wave per (cache block,
// KV head) writes every new token of the block.  K pieces (chunk c, slot t)
// are taken slot-fastest, so the stores of a chunk row are one contiguous
// run; each lane gathers D / 64 dims of every token, so that a block's V^T
// row of a dim (16 slots) is stored at once when the block is written whole
// (element by element for the slots of a partly written block).  The bits
// stored are the plain append's.
template <int DT, int D>
__global__ __launch_bounds__(256) void append_block_kernel(AppendArgs a, AppendBlockPlan p) {
  constexpr int RT = DT == 2 ? 0 : DT;  // new rows: bf16 beside an fp8 cache
  using NE = typename Tr<RT>::Elem;
  using CE = typename Tr<DT>::Elem;
  constexpr int X = Tr<DT>::X;           // elements per K chunk of the cache
  constexpr int NC = D / X;
  constexpr int DPL = D / 64;            // V dims per lane
  static_assert((NC * kBlock) % 64 == 0, "K pieces fill whole passes of the wave");
  const int lane = threadIdx.x & 63;
  const int w = blockIdx.x * kWavesPerGroup + wave_uniform(threadIdx.x >> 6);
  const int unit = w / a.hkv, h = w - unit * a.hkv;
  if (unit >= p.unit_start[p.n_seqs]) return;
  const int j = upper_index(p.unit_start, p.n_seqs, unit);
  const int first = p.pos0[j], end = p.pos0[j] + p.ntok[j];  // new positions [first, end)
  const int b = first / kBlock + (unit - p.unit_start[j]);   // cache block index in the sequence
  const int s0 = max(first, b * kBlock) - b * kBlock;          // its new slots [s0, s1)
  const int s1 = min(end, b * kBlock + kBlock) - b * kBlock;
  const int blk = a.block_tables[(size_t)p.seq[j] * a.mb + b];
  if (blk < 0 || blk >= a.nb) return;
  const size_t head = (size_t)blk * a.hkv + h;
  const size_t rstride = (size_t)a.hkv * D;                    // elements between token rows
  const int row_s0 = p.row0[j] + b * kBlock + s0 - first;      // query row of slot s0
  const NE* kn = reinterpret_cast<const NE*>(a.k_new) + (size_t)h * D;
  const NE* vn = reinterpret_cast<const NE*>(a.v_new) + (size_t)h * D;

  // K: piece (chunk c, slot t) of the block from token row row_s0 + t - s0;
  // all of a lane's loads are issued before its stores
  constexpr int KP = NC * kBlock / 64;  // pieces per lane
  u32x4 kw[KP];
#pragma unroll
  for (int u = 0; u < KP; ++u) {
    const int pc = 64 * u + lane, c = pc / kBlock, t = pc % kBlock;
    const int row = row_s0 + min(max(t, s0), s1 - 1) - s0;  // slots outside [s0, s1) reload a valid row
    kw[u] = *reinterpret_cast<const u32x4*>(kn + (size_t)row * rstride + c * X);
  }
#pragma unroll
  for (int u = 0; u < KP; ++u) {
    const int pc = 64 * u + lane, c = pc / kBlock, t = pc % kBlock;
    if (t < s0 || t >= s1) continue;
    CE* dst = reinterpret_cast<CE*>(a.k_cache) + ((head * NC + c) * kBlock + t) * X;
    if constexpr (DT == 2) {
      float kx[8];
      Tr<0>::unpack(kw[u], kx);
      u32x2 kc = {0u, 0u};
#pragma unroll
      for (int e = 0; e < 8; ++e) kc[e / 4] |= f32_to_e4m3(kx[e] * a.inv_k_scale) << (8 * (e % 4));
      *reinterpret_cast<u32x2*>(dst) = kc;
    } else {
      *reinterpret_cast<u32x4*>(dst) = kw[u];
    }
  }

  // V: this lane's dims d = DPL * lane + i of every new token of the block
  CE vals[kBlock][DPL];
#pragma unroll
  for (int t = 0; t < kBlock; ++t) {
    if (t < s0 || t >= s1) continue;
    const NE* src = vn + (size_t)(row_s0 + t - s0) * rstride + DPL * lane;
#pragma unroll
    for (int i = 0; i < DPL; ++i) {
      if constexpr (DT == 2) {
        vals[t][i] = (uint8_t)f32_to_e4m3(__uint_as_float((unsigned)src[i] << 16) * a.inv_v_scale);
      } else {
        vals[t][i] = src[i];
      }
    }
  }
  CE* vdst = reinterpret_cast<CE*>(a.v_cache) + (head * D + DPL * lane) * kBlock;
  if (s0 == 0 && s1 == kBlock) {
#pragma unroll
    for (int i = 0; i < DPL; ++i) {
      constexpr int PER = 16 / sizeof(CE);  // elements per 16-byte store
#pragma unroll
      for (int q = 0; q < kBlock / PER; ++q) {
        CE piece[PER];
#pragma unroll
        for (int e = 0; e < PER; ++e) piece[e] = vals[q * PER + e][i];
        *reinterpret_cast<u32x4*>(vdst + i * kBlock + q * PER) = __builtin_bit_cast(u32x4, piece);
      }
    }
  } else {
#pragma unroll
    for (int t = 0; t < kBlock; ++t)
      if (t >= s0 && t < s1)
#pragma unroll
        for (int i = 0; i < DPL; ++i) vdst[i * kBlock + t] = vals[t][i];
  }
}

// Rotary embedding of 16-byte chunk c of one head row (rotate-half form):
// element i < half pairs with i + half; with the position's angle row cs
// (cos, sin interleaved per pair), y_i = x_i cos - x_{i+half} sin and
// y_{i+half} = x_{i+half} cos + x_i sin, and elements >= 2*half are copied.
// half is a multiple of the chunk's element count.  Each product and each
// sum is rounded to f32 (no fused multiply-add), then the result to the
// storage type.
template <int DT>
__device__ inline u32x4 rope_chunk(const typename Tr<DT>::Elem* row, int c, int half, const float* cs) {
#pragma clang fp contract(off)
  using T = Tr<DT>;
  constexpr int X = T::X;
  const u32x4 w = *reinterpret_cast<const u32x4*>(row + c * X);
  const int e0 = c * X;
  if (e0 >= 2 * half) return w;
  const bool lo = e0 < half;
  const u32x4 wp = *reinterpret_cast<const u32x4*>(row + (lo ? e0 + half : e0 - half));
  const int j0 = lo ? e0 : e0 - half;
  float x[X], xp[X], y[X];
  T::unpack(w, x);
  T::unpack(wp, xp);
#pragma unroll
  for (int e = 0; e < X; ++e) {
    const float a = x[e] * cs[2 * (j0 + e)];
    const float b = xp[e] * cs[2 * (j0 + e) + 1];
    y[e] = lo ? a - b : a + b;
  }
  return T::pack(y);
}

// Append with the rotary embedding: one wave per new token at position pos.
// The wave rotates the token's query row (all Hq heads, in place), writes
// its rotated key row into the cache and copies its value row, as the plain
// append does.  A head's chunks all fall in one pass of the 64 lanes (D / X
// divides 64), so a pass loads every partner chunk before it stores any.
template <int DT, int D>
__global__ __launch_bounds__(256) void rope_append_kernel(AppendArgs a, AppendPlan p, RopeArgs r) {
  constexpr int RT = DT == 2 ? 0 : DT;  // queries and new rows: bf16 beside an fp8 cache
  using T = Tr<RT>;
  using E = typename T::Elem;
  constexpr int X = T::X;
  constexpr int NC = D / X;
  static_assert(64 % NC == 0, "a head row's chunks fit one pass of the wave");
  const int lane = threadIdx.x & 63;
  const int tok = blockIdx.x * kWavesPerGroup + wave_uniform(threadIdx.x >> 6);
  if (tok >= p.tok_start[p.n_seqs]) return;
  const int j = p.unit ? tok : upper_index(p.tok_start, p.n_seqs, tok);
  const int k = tok - p.tok_start[j];
  const int s = p.seq[j];
  const int t = p.row0[j] + k;
  const int pos = p.pos0[j] + k;
  const float* cs = r.cos_sin + (size_t)pos * r.half * 2;

  E* q = reinterpret_cast<E*>(r.q) + (size_t)t * r.hq * D;
  for (int c0 = 0; c0 < r.hq * NC; c0 += 64) {
    const int ci = c0 + lane;
    if (ci >= r.hq * NC) break;
    const u32x4 y = rope_chunk<RT>(q + (ci / NC) * D, ci % NC, r.half, cs);
    *reinterpret_cast<u32x4*>(q + (ci / NC) * D + (ci % NC) * X) = y;
  }

  const int blk = a.block_tables[(size_t)s * a.mb + pos / kBlock];
  if (blk < 0 || blk >= a.nb) return;
  const int slot = pos % kBlock;
  const E* kn = reinterpret_cast<const E*>(a.k_new) + (size_t)t * a.hkv * D;
  const E* vn = reinterpret_cast<const E*>(a.v_new) + (size_t)t * a.hkv * D;
  for (int ci = lane; ci < a.hkv * NC; ci += 64) {
    const int h = ci / NC, c = ci - h * NC;
    const size_t head = (size_t)blk * a.hkv + h;
    if constexpr (DT == 2) {
      // fp8 cache: the rotated key, rounded to bf16, is quantized like a plain new key
      store_fp8_chunk<D>(a, head, c, slot, rope_chunk<RT>(kn + h * D, c, r.half, cs),
                         *reinterpret_cast<const u32x4*>(vn + h * D + c * X));
      continue;
    }
    *reinterpret_cast<u32x4*>(reinterpret_cast<E*>(a.k_cache) + ((head * NC + c) * kBlock + slot) * X) =
        rope_chunk<RT>(kn + h * D, c, r.half, cs);
    E vv[X];
#pragma unroll
    for (int e = 0; e < X; ++e) vv[e] = vn[h * D + c * X + e];
    E* vc = reinterpret_cast<E*>(a.v_cache) + (head * D + c * X) * kBlock + slot;
#pragma unroll
    for (int e = 0; e < X; ++e) vc[e * kBlock] = vv[e];
  }
}

template <template <int, int> class F, typename... Args>
hipError_t dispatch(int dtype, int head_dim, Args&&... args) {
  if (dtype == 0 && head_dim == 128) return F<0, 128>::run(args...);
  if (dtype == 0 && head_dim == 64) return F<0, 64>::run(args...);
  if (dtype == 1 && head_dim == 128) return F<1, 128>::run(args...);
  if (dtype == 1 && head_dim == 64) return F<1, 64>::run(args...);
  if (dtype == 2 && head_dim == 128) return F<2, 128>::run(args...);
  if (dtype == 2 && head_dim == 64) return F<2, 64>::run(args...);
  return hipErrorInvalidValue;
}

template <int DT, int D>
struct AppendL {
  static hipError_t run(const AppendArgs& a, const AppendPlan& p, hipStream_t stream) {
    const int tokens = p.tok_start[p.n_seqs];
    if (tokens == 0) return hipSuccess;
    hipLaunchKernelGGL((append_kernel<DT, D>), dim3((tokens + kWavesPerGroup - 1) / kWavesPerGroup),
                       dim3(64 * kWavesPerGroup), 0, stream, a, p);
    return hipGetLastError();
  }
};

template <int DT, int D>
struct AppendBlockL {
  static hipError_t run(const AppendArgs& a, const AppendBlockPlan& p, hipStream_t stream) {
    const long waves = (long)p.unit_start[p.n_seqs] * a.hkv;
    if (waves == 0) return hipSuccess;
    hipLaunchKernelGGL((append_block_kernel<DT, D>), dim3((unsigned)((waves + kWavesPerGroup - 1) / kWavesPerGroup)),
                       dim3(64 * kWavesPerGroup), 0, stream, a, p);
    return hipGetLastError();
  }
};

template <int DT, int D>
struct RopeAppendL {
  static hipError_t run(const AppendArgs& a, const AppendPlan& p, const RopeArgs& r, hipStream_t stream) {
    const int tokens = p.tok_start[p.n_seqs];
    if (tokens == 0) return hipSuccess;
    hipLaunchKernelGGL((rope_append_kernel<DT, D>), dim3((tokens + kWavesPerGroup - 1) / kWavesPerGroup),
                       dim3(64 * kWavesPerGroup), 0, stream, a, p, r);
    return hipGetLastError();
  }
};

template <int DT, int D>
struct DecodeL {
  static hipError_t run(const AttnArgs& a, const DecodePlan& p, int n_items, hipStream_t stream) {
    const long units = (long)n_items * a.hkv;
    if (units == 0) return hipSuccess;
    hipLaunchKernelGGL((decode_kernel<DT, D>), dim3((unsigned)((units + kWavesPerGroup - 1) / kWavesPerGroup)),
                       dim3(64 * kWavesPerGroup), 0, stream, a, p);
    return hipGetLastError();
  }
};

template <int DT, int D>
struct MergeL {
  static hipError_t run(const AttnArgs& a, const DecodePlan& p, hipStream_t stream) {
    if (p.n_seqs == 0) return hipSuccess;
    hipLaunchKernelGGL((merge_kernel<DT, D>), dim3(p.n_seqs, (a.hq + kMergeWaves - 1) / kMergeWaves),
                       dim3(64 * kMergeWaves), 0, stream, a, p);
    return hipGetLastError();
  }
};

constexpr int kPrefillWaves = 8;   // waves per bf16 prefill workgroup
constexpr int kPrefillStages = 3;  // LDS ring depth of the bf16 prefill kernel

template <int CT, int D>
hipError_t launch_prefill_mfma(const AttnArgs& a, const PrefillPlan& p, int n_tiles, hipStream_t stream) {
  constexpr size_t lds = 2 * kPrefillStages * 4 * kBlock * D * sizeof(uint16_t);
  auto kern = prefill_mfma_kernel<CT, D, kPrefillWaves, kPrefillStages>;
  // The ring exceeds the default 64 KB of dynamic LDS; raise the limit once
  // per device (each GPU keeps its own function attributes).
  static std::atomic<unsigned long long> ready{0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return hipErrorInvalidDevice;
  const unsigned long long bit = 1ull << (dev & 63);
  if (!(ready.load(std::memory_order_relaxed) & bit)) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    ready.fetch_or(bit, std::memory_order_relaxed);
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)n_tiles * a.hkv), dim3(64 * kPrefillWaves), lds, stream, a, p);
  return hipGetLastError();
}

// Prefill chunks: the MFMA kernel for bf16 and fp8 caches, the generic kernel
// for f32 ones.
template <int DT, int D>
struct PrefillL {
  static hipError_t run(const AttnArgs& a, const PrefillPlan& p, int n_tiles, hipStream_t stream) {
    if (n_tiles == 0) return hipSuccess;
    if constexpr (DT == 0 || DT == 2) {
      return launch_prefill_mfma<DT, D>(a, p, n_tiles, stream);
    } else {
      hipLaunchKernelGGL((prefill_kernel<DT, D>), dim3(n_tiles, a.hkv), dim3(64 * kWavesPerGroup), 0, stream, a, p);
      return hipGetLastError();
    }
  }
};

}  // namespace

hipError_t launch_append(const AppendArgs& a, const AppendPlan& p, int dtype, int head_dim, hipStream_t stream) {
  return dispatch<AppendL>(dtype, head_dim, a, p, stream);
}

hipError_t launch_append_blocks(const AppendArgs& a, const AppendBlockPlan& p, int dtype, int head_dim,
                                hipStream_t stream) {
  return dispatch<AppendBlockL>(dtype, head_dim, a, p, stream);
}

hipError_t launch_rope_append(const AppendArgs& a, const AppendPlan& p, const RopeArgs& r, int dtype, int head_dim,
                              hipStream_t stream) {
  return dispatch<RopeAppendL>(dtype, head_dim, a, p, r, stream);
}

int decode_wave_slots(int dtype, int head_dim) {
  // Concurrent decode waves the device can hold: workgroups per CU at this
  // kernel's register use, times waves per workgroup, times CUs.  Cached per
  // device; 2048 when there is no device to ask.
  static std::atomic<int> cache[64][3][2];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 2048;
  const int di = dtype == 0 ? 0 : dtype == 1 ? 1 : 2, hi = head_dim == 128 ? 0 : 1;
  const int known = cache[dev][di][hi].load(std::memory_order_relaxed);
  if (known > 0) return known;
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) return 2048;
  hipError_t e = hipErrorInvalidValue;
  if (dtype == 0 && head_dim == 128)
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, decode_kernel<0, 128>, 256, 0);
  else if (dtype == 0 && head_dim == 64)
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, decode_kernel<0, 64>, 256, 0);
  else if (dtype == 1 && head_dim == 128)
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, decode_kernel<1, 128>, 256, 0);
  else if (dtype == 1 && head_dim == 64)
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, decode_kernel<1, 64>, 256, 0);
  else if (dtype == 2 && head_dim == 128)
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, decode_kernel<2, 128>, 256, 0);
  else if (dtype == 2 && head_dim == 64)
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, decode_kernel<2, 64>, 256, 0);
  if (e != hipSuccess || per_cu <= 0) return 2048;
  const int slots = per_cu * kWavesPerGroup * cus;
  cache[dev][di][hi].store(slots, std::memory_order_relaxed);
  return slots;
}
hipError_t launch_decode(const AttnArgs& a, const DecodePlan& p, int n_items, int dtype, int head_dim,
                         hipStream_t stream) {
  return dispatch<DecodeL>(dtype, head_dim, a, p, n_items, stream);
}
hipError_t launch_merge(const AttnArgs& a, const DecodePlan& p, int dtype, int head_dim, hipStream_t stream) {
  return dispatch<MergeL>(dtype, head_dim, a, p, stream);
}
template <int DT, int D>
struct PrefillMergeL {
  static hipError_t run(const AttnArgs& a, const PrefillPlan& p, hipStream_t stream) {
    const int rows = p.row_start[p.n_seqs];
    if (rows == 0) return hipSuccess;
    constexpr int heads = kMergeWaves * kPrefillMergeHeadsPerWave;
    hipLaunchKernelGGL((prefill_merge_kernel<DT, D>), dim3(rows, (a.hq + heads - 1) / heads),
                       dim3(64 * kMergeWaves), 0, stream, a, p);
    return hipGetLastError();
  }
};

hipError_t launch_prefill_merge(const AttnArgs& a, const PrefillPlan& p, int dtype, int head_dim,
                                hipStream_t stream) {
  return dispatch<PrefillMergeL>(dtype, head_dim, a, p, stream);
}

hipError_t launch_prefill(const AttnArgs& a, const PrefillPlan& p, int n_tiles, int dtype, int head_dim,
                          hipStream_t stream) {
  return dispatch<PrefillL>(dtype, head_dim, a, p, n_tiles, stream);
}

}  // namespace mpa
