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

#include "mpa_internal.h"

namespace mpa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLn2 = 0.69314718055994530942f;

__device__ inline int wave_uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ inline float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ inline short bf16_bits(float x) { return __builtin_bit_cast(short, (__bf16)x); }

// ---------------------------------------------------------------------------
// Element-type traits.  A "round" of the QK^T product consumes one 16-byte
// chunk of K and of Q per lane: one 16x16x32 bf16 MFMA, or four 16x16x4 f32
// MFMAs.  The PV product consumes 4 tokens of one V^T row per lane: one
// 16x16x16 bf16 MFMA, or four 16x16x4 f32 MFMAs.
template <int DT>
struct Tr;

template <>
struct Tr<0> {  // bf16
  using Elem = uint16_t;
  static constexpr int X = 8;
  using Chunk = bf16x8;
  using VFrag = s16x4;
  using PFrag = s16x4;
  static __device__ inline Chunk load_chunk(const Elem* p) {
    return __builtin_bit_cast(Chunk, *reinterpret_cast<const u32x4*>(p));
  }
  static __device__ inline Chunk zero_chunk() {
    u32x4 z = {0u, 0u, 0u, 0u};
    return __builtin_bit_cast(Chunk, z);
  }
  static __device__ inline f32x4 qk(Chunk k, Chunk q, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(k, q, c, 0, 0, 0);
  }
  static __device__ inline VFrag load_v(const Elem* p) {
    return __builtin_bit_cast(VFrag, *reinterpret_cast<const u32x2*>(p));
  }
  static __device__ inline VFrag keep_first(VFrag v, int nvalid) {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = e < nvalid ? v[e] : (short)0;
    return v;
  }
  static __device__ inline PFrag make_p(f32x4 p) {
    PFrag r;
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = bf16_bits(p[e]);
    return r;
  }
  static __device__ inline f32x4 pv(VFrag v, PFrag p, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(v, p, c, 0, 0, 0);
  }
  static __device__ inline void store4(Elem* dst, f32x4 v) {
    s16x4 r;
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = bf16_bits(v[e]);
    *reinterpret_cast<u32x2*>(dst) = __builtin_bit_cast(u32x2, r);
  }
  static __device__ inline void store1(Elem* dst, float v) { *dst = (uint16_t)bf16_bits(v); }
};

template <>
struct Tr<1> {  // f32
  using Elem = float;
  static constexpr int X = 4;
  using Chunk = f32x4;
  using VFrag = f32x4;
  using PFrag = f32x4;
  static __device__ inline Chunk load_chunk(const Elem* p) { return *reinterpret_cast<const f32x4*>(p); }
  static __device__ inline Chunk zero_chunk() { return f32x4{0.f, 0.f, 0.f, 0.f}; }
  static __device__ inline f32x4 qk(Chunk k, Chunk q, f32x4 c) {
#pragma unroll
    for (int j = 0; j < 4; ++j) c = __builtin_amdgcn_mfma_f32_16x16x4f32(k[j], q[j], c, 0, 0, 0);
    return c;
  }
  static __device__ inline VFrag load_v(const Elem* p) { return *reinterpret_cast<const f32x4*>(p); }
  static __device__ inline VFrag keep_first(VFrag v, int nvalid) {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = e < nvalid ? v[e] : 0.f;
    return v;
  }
  static __device__ inline PFrag make_p(f32x4 p) { return p; }
  static __device__ inline f32x4 pv(VFrag v, PFrag p, f32x4 c) {
#pragma unroll
    for (int j = 0; j < 4; ++j) c = __builtin_amdgcn_mfma_f32_16x16x4f32(v[j], p[j], c, 0, 0, 0);
    return c;
  }
  static __device__ inline void store4(Elem* dst, f32x4 v) { *reinterpret_cast<f32x4*>(dst) = v; }
  static __device__ inline void store1(Elem* dst, float v) { *dst = v; }
};

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
template <int DT, int D>
struct RowState {
  f32x4 acc[D / 16];
  float m;  // running max, log2 units
  float l;  // this lane's part of the running sum
};

template <int DT, int D>
__device__ inline void attend_blocks(const AttnArgs& a, const typename Tr<DT>::Chunk* qf,
                                     const int32_t* bt, int g, int kb_begin, int kb_end, int kend,
                                     int limit, RowState<DT, D>& st, bool& poison) {
  using T = Tr<DT>;
  using E = typename T::Elem;
  constexpr int X = T::X;
  constexpr int R = D / (4 * X);
  constexpr int MT = D / 16;
  const int lane = threadIdx.x & 63;
  const int n = lane & 15, grp = lane >> 4;
  const size_t granule = (size_t)D * kBlock;
  for (int kb = kb_begin; kb < kb_end; ++kb) {
    int blk = bt[kb];
    if (blk < 0 || blk >= a.nb) {
      poison = true;
      blk = 0;
    }
    const size_t base = ((size_t)blk * a.hkv + g) * granule;
    const E* kp = reinterpret_cast<const E*>(a.k_cache) + base;
    const E* vp = reinterpret_cast<const E*>(a.v_cache) + base;
    f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int r = 0; r < R; ++r) s = T::qk(T::load_chunk(kp + ((4 * r + grp) * kBlock + n) * X), qf[r], s);
    typename T::VFrag vf[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) vf[mt] = T::load_v(vp + (16 * mt + n) * kBlock + 4 * grp);
    const int key0 = kb * kBlock + 4 * grp;
    float s2[4];
    float bm = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int key = key0 + i;
      s2[i] = (key <= limit && key < kend) ? s[i] * a.scale_log2 : -INFINITY;
      bm = fmaxf(bm, s2[i]);
    }
    bm = fmaxf(bm, __shfl_xor(bm, 16));
    bm = fmaxf(bm, __shfl_xor(bm, 32));
    const float m_new = fmaxf(st.m, bm);
    // A row with no visible key so far keeps m = -inf; use 0 as the pivot
    // so that exp2 sees -inf - 0 = -inf rather than -inf - -inf = NaN.
    const float pivot = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = exp2_fast(st.m - pivot);
    f32x4 p;
#pragma unroll
    for (int i = 0; i < 4; ++i) p[i] = exp2_fast(s2[i] - pivot);
    st.l = st.l * alpha + ((p[0] + p[1]) + (p[2] + p[3]));
    st.m = m_new;
    const auto pf = T::make_p(p);
    const int nvalid = kend - key0;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const auto v = nvalid < 4 ? T::keep_first(vf[mt], nvalid) : vf[mt];
      st.acc[mt] = T::pv(v, pf, st.acc[mt] * alpha);
    }
  }
}

// ---------------------------------------------------------------------------
// Decode: one wave per (sequence, split, KV head); the G query heads of the
// group are the 16 MFMA columns (columns >= G carry zero queries).
template <int DT, int D>
__global__ __launch_bounds__(256) void decode_kernel(AttnArgs a, DecodePlan p) {
  using T = Tr<DT>;
  using E = typename T::Elem;
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
  const int k0 = split * p.split_tokens;
  const int k1 = min(L, k0 + p.split_tokens);
  const int trow = a.qsl[s];
  const int G = a.hq / a.hkv;
  const int n = lane & 15, grp = lane >> 4;
  const bool head_ok = n < G;
  const int h = g * G + (head_ok ? n : 0);

  const E* q = reinterpret_cast<const E*>(a.q) + ((size_t)trow * a.hq + h) * D;
  typename T::Chunk qf[R];
#pragma unroll
  for (int r = 0; r < R; ++r) qf[r] = head_ok ? T::load_chunk(q + (4 * r + grp) * X) : T::zero_chunk();

  RowState<DT, D> st;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) st.acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  st.m = -INFINITY;
  st.l = 0.f;
  bool poison = false;
  attend_blocks<DT, D>(a, qf, a.block_tables + (size_t)s * a.mb, g, k0 / kBlock,
                       (k1 + kBlock - 1) / kBlock, k1, INT32_MAX, st, poison);

  float l = st.l + __shfl_xor(st.l, 16);
  l += __shfl_xor(l, 32);
  if (!head_ok) return;
  if (nsplit == 1) {
    const float inv = poison ? NAN : 1.f / l;
    E* o = reinterpret_cast<E*>(a.out) + ((size_t)trow * a.hq + h) * D;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) T::store4(o + 16 * mt + 4 * grp, st.acc[mt] * inv);
    if (a.lse && grp == 0) a.lse[(size_t)trow * a.hq + h] = poison ? NAN : (st.m + log2f(l)) * kLn2;
  } else {
    const size_t slot = (size_t)(p.item_base + item) * a.hq + h;
    float* wo = a.ws_o + slot * D;
    const float bad = poison ? NAN : 1.f;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) *reinterpret_cast<f32x4*>(wo + 16 * mt + 4 * grp) = st.acc[mt] * bad;
    if (grp == 0) {
      a.ws_ml[slot * 2] = st.m;
      a.ws_ml[slot * 2 + 1] = l * bad;
    }
  }
}

// Split-K merge: one 64-lane workgroup per (decode sequence, query head).
// With split maxima m_j and sums l_j (log2 units), the row's softmax
// denominator is sum_j l_j 2^(m_j - M) with M = max_j m_j, and its output is
// sum_j acc_j 2^(m_j - M) divided by that denominator.
template <int DT, int D>
__global__ __launch_bounds__(64) void merge_kernel(AttnArgs a, DecodePlan p) {
  using T = Tr<DT>;
  using E = typename T::Elem;
  constexpr int PER = D / 64;
  const int j = blockIdx.x;
  const int h = blockIdx.y;
  if (j >= p.n_seqs) return;
  const int n = p.item_start[j + 1] - p.item_start[j];
  if (n <= 1) return;
  const int s = p.seq[j];
  const size_t base = (size_t)p.item_base + p.item_start[j];
  float M = -INFINITY;
  for (int i = 0; i < n; ++i) M = fmaxf(M, a.ws_ml[((base + i) * a.hq + h) * 2]);
  float lsum = 0.f;
  float o[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) o[e] = 0.f;
  for (int i = 0; i < n; ++i) {
    const size_t slot = (base + i) * a.hq + h;
    const float w = exp2_fast(a.ws_ml[slot * 2] - M);
    lsum += w * a.ws_ml[slot * 2 + 1];
#pragma unroll
    for (int e = 0; e < PER; ++e) o[e] += w * a.ws_o[slot * D + threadIdx.x + 64 * e];
  }
  const int t = a.qsl[s];
  E* out = reinterpret_cast<E*>(a.out) + ((size_t)t * a.hq + h) * D;
  const float inv = 1.f / lsum;
#pragma unroll
  for (int e = 0; e < PER; ++e) T::store1(out + threadIdx.x + 64 * e, o[e] * inv);
  if (a.lse && threadIdx.x == 0) a.lse[(size_t)t * a.hq + h] = (M + log2f(lsum)) * kLn2;
}

// ---------------------------------------------------------------------------
// Prefill chunks: one workgroup per (sequence, query tile, KV head).  The
// tile's 64 (token, head) rows are the 16 columns of each of the 4 waves;
// row r is token r / G of the tile and head r % G of the group.
template <int DT, int D>
__global__ __launch_bounds__(256) void prefill_kernel(AttnArgs a, PrefillPlan p) {
  using T = Tr<DT>;
  using E = typename T::Elem;
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
  const int i_raw = first_tok + row / G;
  const bool row_ok = i_raw < C;
  const int i = row_ok ? i_raw : C - 1;
  const int h = g * G + row % G;
  const int last_tok = min(first_tok + (wave * 16 + 15) / G, C - 1);
  const int kend = P + last_tok + 1;  // keys this wave needs

  const E* q = reinterpret_cast<const E*>(a.q) + ((size_t)(t0 + i) * a.hq + h) * D;
  typename T::Chunk qf[R];
#pragma unroll
  for (int r = 0; r < R; ++r) qf[r] = T::load_chunk(q + (4 * r + grp) * X);

  RowState<DT, D> st;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) st.acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  st.m = -INFINITY;
  st.l = 0.f;
  bool poison = false;
  attend_blocks<DT, D>(a, qf, a.block_tables + (size_t)s * a.mb, g, 0, (kend + kBlock - 1) / kBlock,
                       kend, P + i, st, poison);

  float l = st.l + __shfl_xor(st.l, 16);
  l += __shfl_xor(l, 32);
  if (!row_ok) return;
  const float inv = poison ? NAN : 1.f / l;
  E* o = reinterpret_cast<E*>(a.out) + ((size_t)(t0 + i) * a.hq + h) * D;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) T::store4(o + 16 * mt + 4 * grp, st.acc[mt] * inv);
  if (a.lse && grp == 0) a.lse[(size_t)(t0 + i) * a.hq + h] = poison ? NAN : (st.m + log2f(l)) * kLn2;
}

// ---------------------------------------------------------------------------
// Append: one thread per 16-byte chunk of one new (token, KV head) key row;
// the same thread copies the matching X value elements.
template <int DT, int D>
__global__ __launch_bounds__(256) void append_kernel(AppendArgs a) {
  using T = Tr<DT>;
  using E = typename T::Elem;
  constexpr int X = T::X;
  constexpr int NC = D / X;
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  const long total = (long)a.total_q * a.hkv * NC;
  if (idx >= total) return;
  const int c = (int)(idx % NC);
  const long th = idx / NC;
  const int h = (int)(th % a.hkv);
  const int t = (int)(th / a.hkv);
  const int s = upper_index(a.qsl, a.num_seqs, t);
  const int pos = a.seq_lens[s] - (a.qsl[s + 1] - a.qsl[s]) + (t - a.qsl[s]);
  const int blk = a.block_tables[(size_t)s * a.mb + pos / kBlock];
  if (blk < 0 || blk >= a.nb) return;
  const int slot = pos % kBlock;
  const size_t head = (size_t)blk * a.hkv + h;
  const E* kn = reinterpret_cast<const E*>(a.k_new) + ((size_t)t * a.hkv + h) * D + c * X;
  E* kc = reinterpret_cast<E*>(a.k_cache) + ((head * NC + c) * kBlock + slot) * X;
  *reinterpret_cast<u32x4*>(kc) = *reinterpret_cast<const u32x4*>(kn);
  const E* vn = reinterpret_cast<const E*>(a.v_new) + ((size_t)t * a.hkv + h) * D + c * X;
  E* vc = reinterpret_cast<E*>(a.v_cache) + (head * D + c * X) * kBlock + slot;
#pragma unroll
  for (int e = 0; e < X; ++e) vc[e * kBlock] = vn[e];
}

template <template <int, int> class F, typename... Args>
hipError_t dispatch(int dtype, int head_dim, Args&&... args) {
  if (dtype == 0 && head_dim == 128) return F<0, 128>::run(args...);
  if (dtype == 0 && head_dim == 64) return F<0, 64>::run(args...);
  if (dtype == 1 && head_dim == 128) return F<1, 128>::run(args...);
  if (dtype == 1 && head_dim == 64) return F<1, 64>::run(args...);
  return hipErrorInvalidValue;
}

template <int DT, int D>
struct AppendL {
  static hipError_t run(const AppendArgs& a, hipStream_t stream) {
    const long total = (long)a.total_q * a.hkv * (D / Tr<DT>::X);
    if (total == 0) return hipSuccess;
    hipLaunchKernelGGL((append_kernel<DT, D>), dim3((unsigned)((total + 255) / 256)), dim3(256), 0, stream, a);
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
    hipLaunchKernelGGL((merge_kernel<DT, D>), dim3(p.n_seqs, a.hq), dim3(64), 0, stream, a, p);
    return hipGetLastError();
  }
};

template <int DT, int D>
struct PrefillL {
  static hipError_t run(const AttnArgs& a, const PrefillPlan& p, int n_tiles, hipStream_t stream) {
    if (n_tiles == 0) return hipSuccess;
    hipLaunchKernelGGL((prefill_kernel<DT, D>), dim3(n_tiles, a.hkv), dim3(64 * kWavesPerGroup), 0, stream, a, p);
    return hipGetLastError();
  }
};

}  // namespace

hipError_t launch_append(const AppendArgs& a, int dtype, int head_dim, hipStream_t stream) {
  return dispatch<AppendL>(dtype, head_dim, a, stream);
}
hipError_t launch_decode(const AttnArgs& a, const DecodePlan& p, int n_items, int dtype, int head_dim,
                         hipStream_t stream) {
  return dispatch<DecodeL>(dtype, head_dim, a, p, n_items, stream);
}
hipError_t launch_merge(const AttnArgs& a, const DecodePlan& p, int dtype, int head_dim, hipStream_t stream) {
  return dispatch<MergeL>(dtype, head_dim, a, p, stream);
}
hipError_t launch_prefill(const AttnArgs& a, const PrefillPlan& p, int n_tiles, int dtype, int head_dim,
                          hipStream_t stream) {
  return dispatch<PrefillL>(dtype, head_dim, a, p, n_tiles, stream);
}

}  // namespace mpa
