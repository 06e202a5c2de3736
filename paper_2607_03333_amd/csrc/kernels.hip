// gfx950 (MI355X, CDNA4) kernels of the forked-decode hot path.
//
//  * attn_bf16 / attn_f32: partial attention of one work item's token range
//    for up to RT 16-row tiles of query rows (split-K). A work item is either
//    a fork group's shared prefix, read once for every member's rows
//    (Section 4.1: probes reuse the main thread's prefix KV), or one
//    thread's private range, where verify rows apply the causal rule over
//    the drafts (Section 4.3). Q.K^T and P.V run on MFMA with fp32
//    accumulation; K and V stream from HBM with 16-byte loads straight into
//    the MFMA operand registers.
//  * merge: log-sum-exp merge of an output row's partials (DPP wave
//    reductions), written in the input dtype, plus the row's lse.
//  * argmax_chunks + accept: greedy token of every verify row (lowest index of
//    the row maximum) and the longest draft prefix equal to the greedy tokens
//    (Section 4.3, steps 2-3).
//  * kv_write / kv_copy: token scatter into the paged pools and the copy of
//    copy-on-write (setup work, not on the timed path).
#include <hip/hip_runtime.h>

#include <climits>
#include <cstdint>

#include "kernels.h"

namespace spork {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kLn2 = 0.693147180559945309f;

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// --------------------------------------------------------------------------
// Wave-wide reductions with DPP: butterflies inside each 16-lane row
// (quad permutes, half-row and row mirrors), then the row broadcasts 15 and
// 31 carry the partial results across rows; lane 63 ends with the total.
// --------------------------------------------------------------------------
template <int kCtrl, int kRowMask>
__device__ __forceinline__ float dpp_mov(float ident, float x) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, ident), __builtin_bit_cast(int, x),
                                         kCtrl, kRowMask, 0xF, false));
}

template <typename Op>
__device__ __forceinline__ float wave_reduce(float x, float ident, Op op) {
  x = op(x, dpp_mov<0xB1, 0xF>(ident, x));   // quad_perm [1,0,3,2]
  x = op(x, dpp_mov<0x4E, 0xF>(ident, x));   // quad_perm [2,3,0,1]
  x = op(x, dpp_mov<0x141, 0xF>(ident, x));  // row_half_mirror
  x = op(x, dpp_mov<0x140, 0xF>(ident, x));  // row_mirror
  x = op(x, dpp_mov<0x142, 0xA>(ident, x));  // row_bcast:15 into rows 1 and 3
  x = op(x, dpp_mov<0x143, 0xC>(ident, x));  // row_bcast:31 into rows 2 and 3
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 63));
}

__device__ __forceinline__ float wave_max(float x) {
  return wave_reduce(x, kNegInf, [](float a, float b) { return fmaxf(a, b); });
}
__device__ __forceinline__ float wave_sum(float x) {
  return wave_reduce(x, 0.0f, [](float a, float b) { return a + b; });
}

// --------------------------------------------------------------------------
// Online softmax step shared by both attention kernels. `sv` holds this
// lane's 8 base-2 scores (query row = lane % 16, tokens chosen by the caller;
// the 4 lanes with the same lane % 16 together hold 32 tokens). Updates the
// lane's running max / partial sum and returns the probabilities and the
// rescale factor for the accumulator.
// --------------------------------------------------------------------------
__device__ __forceinline__ float softmax_step(float (&sv)[8], float& m, float& l) {
  float mx = sv[0];
#pragma unroll
  for (int j = 1; j < 8; ++j) mx = fmaxf(mx, sv[j]);
  mx = fmaxf(mx, __shfl_xor(mx, 16));
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  const float mn = fmaxf(m, mx);
  const float mu = mn == kNegInf ? 0.0f : mn;  // rows with nothing visible yet stay at zero
  const float alpha = exp2_fast(m - mu);
  float ps = 0.0f;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    sv[j] = exp2_fast(sv[j] - mu);
    ps += sv[j];
  }
  l = l * alpha + ps;
  m = mn;
  return alpha;
}

__device__ __forceinline__ int wave_min_int(int x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = min(x, __shfl_xor(x, o));
  return x;
}

// --------------------------------------------------------------------------
// bf16 partial attention: RT row tiles, head dim D, block size BS.
//
// Per 32-token tile and row tile, with r16 = lane % 16 and g = lane / 16:
//   S^T = K Q^T via v_mfma_f32_16x16x32_bf16: A-row r16 of half hh is token
//   tb + 8*(r16/4) + 4*hh + r16%4, so the lane receives scores of query row
//   r16 for tokens tb + 8g + j (j = 0..7, halves concatenated).
//   O^T += V^T P^T via the same MFMA: A = V^T (channel 16*dt + r16, tokens
//   tb + 8g .. +7: one 16-byte load from the channel-major V block),
//   B = P^T (the lane's own 8 probabilities). The accumulator gives the lane
//   query row r16 at channels 16*dt + 4g + i, so the rescale is lane-local.
//   The contraction slot of channel d in Q.K is (k-step d/32, lane group
//   (d%32)/8, element d%8) on both operands.
// --------------------------------------------------------------------------
template <int RT, int D, int BS>
__global__ void __launch_bounds__(64) attn_bf16(AttnArgs a) {
  static_assert(D % 32 == 0 && (BS == 16 || BS == 32 || BS == 64), "unsupported shape");
  constexpr int KS = D / 32;
  constexpr int DT = D / 16;
  const WaveDesc w = a.waves[blockIdx.x];
  if (w.item < 0) return;
  const ItemDesc it = a.items[w.item];
  const int lane = threadIdx.x, r16 = lane & 15, g = lane >> 4;
  const uint16_t* __restrict__ qg = static_cast<const uint16_t*>(a.q);
  const uint16_t* __restrict__ kc = static_cast<const uint16_t*>(a.k_cache);
  const uint16_t* __restrict__ vc = static_cast<const uint16_t*>(a.v_cache);
  const int32_t* __restrict__ table = a.tables + it.table_off;
  const int nb = it.n_blocks;
  const size_t head = static_cast<size_t>(it.kv_head);
  const size_t hkv = static_cast<size_t>(a.hkv);
  const int ntiles = (w.nrows + 15) >> 4;

  bf16x8 qop[RT][KS];
  int hz[RT];
#pragma unroll
  for (int t = 0; t < RT; ++t) {
    const int i = t * 16 + r16;
    if (i < w.nrows) {
      const RowDesc rd = a.rows[it.row_off + w.row0 + i];
      hz[t] = rd.horizon;
      const uint4* qp = reinterpret_cast<const uint4*>(qg + static_cast<size_t>(rd.qidx) * D);
#pragma unroll
      for (int s = 0; s < KS; ++s) qop[t][s] = as_bf16x8(qp[4 * s + g]);
    } else {
      hz[t] = INT_MAX;  // padding row: zero query, never written
#pragma unroll
      for (int s = 0; s < KS; ++s) qop[t][s] = as_bf16x8(make_uint4(0, 0, 0, 0));
    }
  }
  int hmin = INT_MAX;
#pragma unroll
  for (int t = 0; t < RT; ++t) hmin = min(hmin, hz[t]);
  hmin = wave_min_int(hmin);

  float m[RT], l[RT];
  f32x4 o[RT][DT];
#pragma unroll
  for (int t = 0; t < RT; ++t) {
    m[t] = kNegInf;
    l[t] = 0.0f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[t][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // Physical block of the tile's j-th block (clamped to the table: positions
  // past the range are masked, and their V is zeroed before use).
  auto blk = [&](int tb, int j) {
    int bi = tb / BS + j;
    bi = bi < nb ? bi : nb - 1;
    return static_cast<size_t>(table[bi]);
  };
  auto load_tile = [&](int tb, bf16x8 (&kop)[2][KS], bf16x8 (&vop)[DT]) {
    const size_t b0 = blk(tb, 0);
    const size_t b1 = BS == 16 ? blk(tb, 1) : b0;
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int tk = 8 * (r16 >> 2) + 4 * hh + (r16 & 3);  // 0..31 within the tile
      const size_t b = (BS == 16 && tk >= 16) ? b1 : b0;
      const int off = (tb + tk) % BS;
      const uint4* kp = reinterpret_cast<const uint4*>(
          kc + ((b * hkv + head) * BS + off) * D);
#pragma unroll
      for (int s = 0; s < KS; ++s) kop[hh][s] = as_bf16x8(kp[4 * s + g]);
    }
    const size_t bv = (BS == 16 && g >= 2) ? b1 : b0;
    const int offv = (tb + 8 * g) % BS;
    const uint16_t* vp = vc + (bv * hkv + head) * (static_cast<size_t>(D) * BS) + offv;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
      vop[dt] = as_bf16x8(*reinterpret_cast<const uint4*>(vp + static_cast<size_t>(16 * dt + r16) * BS));
  };

  const float c = a.scale_log2;
  int tb = w.tok_lo & ~(kTileTokens - 1);
  bf16x8 kA[2][KS], vA[DT];
  load_tile(tb, kA, vA);
  for (; tb < w.tok_hi; tb += kTileTokens) {
    bf16x8 kB[2][KS], vB[DT];
    const bool more = tb + kTileTokens < w.tok_hi;
    if (more) load_tile(tb + kTileTokens, kB, vB);
    const bool edge = tb < w.tok_lo || tb + kTileTokens > w.tok_hi || tb + kTileTokens - 1 > hmin;
    if (tb + kTileTokens > w.tok_hi) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (tb + 8 * g + j >= w.tok_hi) {
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) vA[dt][j] = static_cast<__bf16>(0.0f);
        }
      }
    }
#pragma unroll
    for (int t = 0; t < RT; ++t) {
      if (t < ntiles) {
        f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kA[0][s], qop[t][s], s0, 0, 0, 0);
          s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kA[1][s], qop[t][s], s1, 0, 0, 0);
        }
        float sv[8] = {s0[0] * c, s0[1] * c, s0[2] * c, s0[3] * c,
                       s1[0] * c, s1[1] * c, s1[2] * c, s1[3] * c};
        if (edge) {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int tk = tb + 8 * g + j;
            if (tk < w.tok_lo || tk >= w.tok_hi || tk > hz[t]) sv[j] = kNegInf;
          }
        }
        const float alpha = softmax_step(sv, m[t], l[t]);
        bf16x8 pop;
#pragma unroll
        for (int j = 0; j < 8; ++j) pop[j] = static_cast<__bf16>(sv[j]);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          o[t][dt] *= alpha;
          o[t][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vA[dt], pop, o[t][dt], 0, 0, 0);
        }
      }
    }
    if (more) {
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int s = 0; s < KS; ++s) kA[hh][s] = kB[hh][s];
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) vA[dt] = vB[dt];
    }
  }

#pragma unroll
  for (int t = 0; t < RT; ++t) {
    if (t < ntiles) {
      float lt = l[t] + __shfl_xor(l[t], 16);
      lt += __shfl_xor(lt, 32);
      const int i = t * 16 + r16;
      if (i < w.nrows) {
        const size_t pr = static_cast<size_t>(w.partial + i);
        if (g == 0) {
          a.part_ml[2 * pr] = m[t];
          a.part_ml[2 * pr + 1] = lt;
        }
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          *reinterpret_cast<f32x4*>(a.part_o + pr * D + 16 * dt + 4 * g) = o[t][dt];
      }
    }
  }
}

// --------------------------------------------------------------------------
// fp32 partial attention (full-precision v_mfma_f32_16x16x4_f32).
//   Scores: half hh of the tile has A-row r16 = token tb + 16*hh + r16, and the
//   contraction slot of channel d is (k-step d/4, lane group d%4); the lane
//   receives query row r16 for tokens tb + 16*hh + 4g + i.
//   P.V: one MFMA per (hh, i) over the 4 tokens tb + 16*hh + 4g' + i
//   (g' = 0..3): A = V^T (channel 16*dt + r16, the lane's token), B = the
//   lane's own probability. Accumulator layout as in the bf16 kernel.
// --------------------------------------------------------------------------
template <int RT, int D, int BS>
__global__ void __launch_bounds__(64) attn_f32(AttnArgs a) {
  static_assert(D % 16 == 0 && (BS == 16 || BS == 32 || BS == 64), "unsupported shape");
  constexpr int KS = D / 4;
  constexpr int DT = D / 16;
  const WaveDesc w = a.waves[blockIdx.x];
  if (w.item < 0) return;
  const ItemDesc it = a.items[w.item];
  const int lane = threadIdx.x, r16 = lane & 15, g = lane >> 4;
  const float* __restrict__ qg = static_cast<const float*>(a.q);
  const float* __restrict__ kc = static_cast<const float*>(a.k_cache);
  const float* __restrict__ vc = static_cast<const float*>(a.v_cache);
  const int32_t* __restrict__ table = a.tables + it.table_off;
  const int nb = it.n_blocks;
  const size_t head = static_cast<size_t>(it.kv_head);
  const size_t hkv = static_cast<size_t>(a.hkv);
  const int ntiles = (w.nrows + 15) >> 4;

  float qop[RT][KS];
  int hz[RT];
#pragma unroll
  for (int t = 0; t < RT; ++t) {
    const int i = t * 16 + r16;
    if (i < w.nrows) {
      const RowDesc rd = a.rows[it.row_off + w.row0 + i];
      hz[t] = rd.horizon;
      const float* qp = qg + static_cast<size_t>(rd.qidx) * D;
#pragma unroll
      for (int s = 0; s < KS; ++s) qop[t][s] = qp[4 * s + g];
    } else {
      hz[t] = INT_MAX;
#pragma unroll
      for (int s = 0; s < KS; ++s) qop[t][s] = 0.0f;
    }
  }
  int hmin = INT_MAX;
#pragma unroll
  for (int t = 0; t < RT; ++t) hmin = min(hmin, hz[t]);
  hmin = wave_min_int(hmin);

  float m[RT], l[RT];
  f32x4 o[RT][DT];
#pragma unroll
  for (int t = 0; t < RT; ++t) {
    m[t] = kNegInf;
    l[t] = 0.0f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[t][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  auto blk = [&](int tb, int j) {
    int bi = tb / BS + j;
    bi = bi < nb ? bi : nb - 1;
    return static_cast<size_t>(table[bi]);
  };

  const float c = a.scale_log2;
  for (int tb = w.tok_lo & ~(kTileTokens - 1); tb < w.tok_hi; tb += kTileTokens) {
    const size_t b0 = blk(tb, 0);
    const size_t b1 = BS == 16 ? blk(tb, 1) : b0;
    float kop[2][KS];
    f32x4 vop[2][DT];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const size_t b = (BS == 16 && hh == 1) ? b1 : b0;
      const int offk = (tb + 16 * hh + r16) % BS;
      const float* kp = kc + ((b * hkv + head) * BS + offk) * D;
#pragma unroll
      for (int s = 0; s < KS; ++s) kop[hh][s] = kp[4 * s + g];
      const int offv = (tb + 16 * hh + 4 * g) % BS;
      const float* vp = vc + (b * hkv + head) * (static_cast<size_t>(D) * BS) + offv;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        f32x4 v = *reinterpret_cast<const f32x4*>(vp + static_cast<size_t>(16 * dt + r16) * BS);
        if (tb + kTileTokens > w.tok_hi) {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (tb + 16 * hh + 4 * g + i >= w.tok_hi) v[i] = 0.0f;
        }
        vop[hh][dt] = v;
      }
    }
    const bool edge = tb < w.tok_lo || tb + kTileTokens > w.tok_hi || tb + kTileTokens - 1 > hmin;
#pragma unroll
    for (int t = 0; t < RT; ++t) {
      if (t < ntiles) {
        f32x4 sc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int s = 0; s < KS; ++s)
            sc[hh] = __builtin_amdgcn_mfma_f32_16x16x4f32(kop[hh][s], qop[t][s], sc[hh], 0, 0, 0);
        float sv[8];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
#pragma unroll
          for (int i = 0; i < 4; ++i) sv[4 * hh + i] = sc[hh][i] * c;
        if (edge) {
#pragma unroll
          for (int hh = 0; hh < 2; ++hh)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int tk = tb + 16 * hh + 4 * g + i;
              if (tk < w.tok_lo || tk >= w.tok_hi || tk > hz[t]) sv[4 * hh + i] = kNegInf;
            }
        }
        const float alpha = softmax_step(sv, m[t], l[t]);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          o[t][dt] *= alpha;
#pragma unroll
          for (int hh = 0; hh < 2; ++hh)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              o[t][dt] = __builtin_amdgcn_mfma_f32_16x16x4f32(vop[hh][dt][i], sv[4 * hh + i], o[t][dt], 0, 0, 0);
        }
      }
    }
  }

#pragma unroll
  for (int t = 0; t < RT; ++t) {
    if (t < ntiles) {
      float lt = l[t] + __shfl_xor(l[t], 16);
      lt += __shfl_xor(lt, 32);
      const int i = t * 16 + r16;
      if (i < w.nrows) {
        const size_t pr = static_cast<size_t>(w.partial + i);
        if (g == 0) {
          a.part_ml[2 * pr] = m[t];
          a.part_ml[2 * pr + 1] = lt;
        }
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          *reinterpret_cast<f32x4*>(a.part_o + pr * D + 16 * dt + 4 * g) = o[t][dt];
      }
    }
  }
}

// --------------------------------------------------------------------------
// Log-sum-exp merge: one wave per output (query row x query head).
//   M = max m_i, L = sum 2^(m_i - M) l_i, O = sum 2^(m_i - M) o_i / L,
//   lse = (M + log2 L) ln 2. Partials with nothing visible (m = -inf, l = 0)
//   add nothing.
// --------------------------------------------------------------------------
template <int D, typename OutT>
__global__ void __launch_bounds__(256) merge_kernel(AttnArgs a) {
  constexpr int PER = D / 64;
  const int o = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (o >= a.n_out) return;
  const int beg = a.merge_off[o], end = a.merge_off[o + 1];
  float mx = kNegInf;
  for (int c = beg + lane; c < end; c += 64) mx = fmaxf(mx, a.part_ml[2 * a.merge_ids[c]]);
  mx = wave_max(mx);
  const float mu = mx == kNegInf ? 0.0f : mx;
  float sum = 0.0f;
  for (int c = beg + lane; c < end; c += 64) {
    const int id = a.merge_ids[c];
    sum += exp2_fast(a.part_ml[2 * id] - mu) * a.part_ml[2 * id + 1];
  }
  sum = wave_sum(sum);
  float acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.0f;
  for (int c = beg; c < end; ++c) {
    const int id = a.merge_ids[c];
    const float wgt = exp2_fast(a.part_ml[2 * id] - mu);
    const float* po = a.part_o + static_cast<size_t>(id) * D + lane * PER;
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] += wgt * po[e];
  }
  const float inv = sum > 0.0f ? 1.0f / sum : 0.0f;
  OutT* out = static_cast<OutT*>(a.out) + static_cast<size_t>(o) * D + lane * PER;
#pragma unroll
  for (int e = 0; e < PER; ++e) out[e] = static_cast<OutT>(acc[e] * inv);
  if (lane == 0 && a.lse != nullptr)
    a.lse[o] = sum > 0.0f ? (mu + __log2f(sum)) * kLn2 : kNegInf;
}

// --------------------------------------------------------------------------
// Greedy argmax, first pass: the best (value, index) of one chunk of a row.
// Each thread scans its elements in increasing index order keeping the first
// strict maximum; chunks and threads combine through the 64-bit key
// (order-preserving value bits << 32) | (0xFFFFFFFF - index), whose maximum
// is the largest value at the lowest index. -0 is keyed as +0.
// --------------------------------------------------------------------------
__device__ __forceinline__ uint64_t argmax_key(float v, int idx) {
  if (idx == INT_MAX) return 0;
  uint32_t u = __float_as_uint(v == 0.0f ? 0.0f : v);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return (static_cast<uint64_t>(u) << 32) | (0xFFFFFFFFu - static_cast<uint32_t>(idx));
}

__device__ __forceinline__ float load_f(const float* p, int i) { return p[i]; }
__device__ __forceinline__ float load_f(const uint16_t* p, int i) {
  return __uint_as_float(static_cast<uint32_t>(p[i]) << 16);
}

template <typename T>
__global__ void __launch_bounds__(256) argmax_chunks(AcceptArgs a) {
  constexpr int VEC = 16 / sizeof(T);
  const int row = blockIdx.x / a.chunks, c = blockIdx.x % a.chunks;
  const T* x = static_cast<const T*>(a.logits) + static_cast<size_t>(row) * a.vocab;
  float best = kNegInf;
  int bidx = INT_MAX;
  const bool vec_ok = (a.vocab % VEC) == 0 && (reinterpret_cast<uintptr_t>(a.logits) & 15) == 0;
  if (vec_ok) {
    const int nv = a.vocab / VEC;
    const int lo = static_cast<int>(static_cast<int64_t>(nv) * c / a.chunks);
    const int hi = static_cast<int>(static_cast<int64_t>(nv) * (c + 1) / a.chunks);
    for (int v = lo + static_cast<int>(threadIdx.x); v < hi; v += 256) {
      const uint4 u = reinterpret_cast<const uint4*>(x)[v];
      const T* e = reinterpret_cast<const T*>(&u);
#pragma unroll
      for (int j = 0; j < VEC; ++j) {
        const float val = load_f(e, j);
        if (val > best || bidx == INT_MAX) {
          best = val;
          bidx = v * VEC + j;
        }
      }
    }
  } else {
    const int lo = static_cast<int>(static_cast<int64_t>(a.vocab) * c / a.chunks);
    const int hi = static_cast<int>(static_cast<int64_t>(a.vocab) * (c + 1) / a.chunks);
    for (int i = lo + static_cast<int>(threadIdx.x); i < hi; i += 256) {
      const float val = load_f(x, i);
      if (val > best || bidx == INT_MAX) {
        best = val;
        bidx = i;
      }
    }
  }
  uint64_t key = argmax_key(best, bidx);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const uint64_t other = __shfl_xor(key, o);
    key = other > key ? other : key;
  }
  __shared__ uint64_t wk[4];
  if ((threadIdx.x & 63) == 0) wk[threadIdx.x >> 6] = key;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t k = wk[0];
    for (int i = 1; i < 4; ++i) k = wk[i] > k ? wk[i] : k;
    a.keys[static_cast<size_t>(row) * a.chunks + c] = k;
  }
}

// Accept: per verify thread, combine the chunk keys of its K+1 rows, then the
// first draft that differs from the greedy token ends the accepted prefix.
__global__ void __launch_bounds__(64) accept_kernel(AcceptArgs a) {
  extern __shared__ int greedy[];
  const int s = blockIdx.x, kd = a.k_drafts;
  for (int r = threadIdx.x; r <= kd; r += 64) {
    const uint64_t* kp = a.keys + static_cast<size_t>(s * (kd + 1) + r) * a.chunks;
    uint64_t best = 0;
    for (int c = 0; c < a.chunks; ++c) best = kp[c] > best ? kp[c] : best;
    const int idx = static_cast<int>(0xFFFFFFFFu - static_cast<uint32_t>(best));
    greedy[r] = idx;
    if (a.argmax_out != nullptr) a.argmax_out[s * (kd + 1) + r] = idx;
  }
  __syncthreads();
  // first mismatch via a ballot over the draft positions
  int first = kd;
  for (int base = 0; base < kd; base += 64) {
    const int r = base + static_cast<int>(threadIdx.x);
    const bool miss = r < kd && greedy[r] != a.drafts[static_cast<size_t>(s) * kd + r];
    const uint64_t bal = __ballot(miss);
    if (bal != 0) {
      first = base + __builtin_ctzll(bal);
      break;
    }
  }
  if (threadIdx.x == 0) {
    a.accept_len[s] = first;
    a.next_token[s] = greedy[first];
  }
}

// --------------------------------------------------------------------------
// Setup kernels.
// --------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256) kv_write_kernel(int hkv, int D, int BS, int64_t num_slots, T* kc,
                                                       T* vc, const int64_t* slots, const T* kn,
                                                       const T* vn, int n, int* bad) {
  constexpr int VEC = 16 / sizeof(T);
  const int per_tok = hkv * (D / VEC);
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= static_cast<int64_t>(n) * per_tok) return;
  const int i = static_cast<int>(idx / per_tok);
  const int rem = static_cast<int>(idx % per_tok);
  const int h = rem / (D / VEC), cchunk = rem % (D / VEC);
  const int64_t slot = slots[i];
  if (slot < 0 || slot >= num_slots) {
    if (rem == 0 && bad != nullptr) atomicAdd(bad, 1);
    return;
  }
  const int64_t b = slot / BS, off = slot % BS;
  const size_t src = (static_cast<size_t>(i) * hkv + h) * D + static_cast<size_t>(cchunk) * VEC;
  *reinterpret_cast<uint4*>(kc + ((static_cast<size_t>(b) * hkv + h) * BS + off) * D + cchunk * VEC) =
      *reinterpret_cast<const uint4*>(kn + src);
  const T* vs = vn + src;
  T* vd = vc + (static_cast<size_t>(b) * hkv + h) * static_cast<size_t>(D) * BS + off;
#pragma unroll
  for (int e = 0; e < VEC; ++e) vd[static_cast<size_t>(cchunk * VEC + e) * BS] = vs[e];
}

template <typename T>
__global__ void __launch_bounds__(256) kv_copy_kernel(int hkv, int D, int BS, T* kc, T* vc, int src, int dst,
                                                      int nv) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= static_cast<int64_t>(hkv) * nv * D) return;
  const int h = static_cast<int>(idx / (static_cast<int64_t>(nv) * D));
  const int rem = static_cast<int>(idx % (static_cast<int64_t>(nv) * D));
  const int off = rem / D, d = rem % D;
  const size_t ks = ((static_cast<size_t>(src) * hkv + h) * BS + off) * D + d;
  const size_t kd = ((static_cast<size_t>(dst) * hkv + h) * BS + off) * D + d;
  kc[kd] = kc[ks];
  const size_t vs = ((static_cast<size_t>(src) * hkv + h) * D + d) * BS + off;
  const size_t vd = ((static_cast<size_t>(dst) * hkv + h) * D + d) * BS + off;
  vc[vd] = vc[vs];
}

// --------------------------------------------------------------------------
// Dispatch tables.
// --------------------------------------------------------------------------
typedef void (*AttnKernel)(AttnArgs);

template <int D, int BS>
AttnKernel pick_bf16(int rt) {
  switch (rt) {
    case 1: return attn_bf16<1, D, BS>;
    case 2: return attn_bf16<2, D, BS>;
    case 3: return attn_bf16<3, D, BS>;
    case 4: return attn_bf16<4, D, BS>;
    default: return nullptr;
  }
}

template <int D, int BS>
AttnKernel pick_f32(int rt) {
  switch (rt) {
    case 1: return attn_f32<1, D, BS>;
    case 2: return attn_f32<2, D, BS>;
    case 3: return attn_f32<3, D, BS>;
    case 4: return attn_f32<4, D, BS>;
    default: return nullptr;
  }
}

AttnKernel pick_attention(int32_t dtype, int32_t d, int32_t bs, int32_t rt) {
  if (dtype == 1 && d == 128) {
    if (bs == 16) return pick_bf16<128, 16>(rt);
    if (bs == 32) return pick_bf16<128, 32>(rt);
  }
  if (dtype == 0) {
    if (d == 64 && bs == 16) return pick_f32<64, 16>(rt);
    if (d == 64 && bs == 32) return pick_f32<64, 32>(rt);
    if (d == 128 && bs == 16) return pick_f32<128, 16>(rt);
    if (d == 128 && bs == 32) return pick_f32<128, 32>(rt);
  }
  return nullptr;
}

}  // namespace

bool attention_supported(int32_t dtype, int32_t head_dim, int32_t block_size, int32_t row_tiles) {
  return pick_attention(dtype, head_dim, block_size, row_tiles) != nullptr;
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t stream) {
  AttnKernel k = pick_attention(a.dtype, a.head_dim, a.block_size, a.row_tiles);
  if (k == nullptr) return hipErrorInvalidValue;
  if (a.n_waves > 0) hipLaunchKernelGGL(k, dim3(a.n_waves), dim3(64), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int blocks = (a.n_out + 3) / 4;
  if (blocks > 0) {
    if (a.dtype == 1 && a.head_dim == 128)
      hipLaunchKernelGGL((merge_kernel<128, __bf16>), dim3(blocks), dim3(256), 0, stream, a);
    else if (a.dtype == 0 && a.head_dim == 128)
      hipLaunchKernelGGL((merge_kernel<128, float>), dim3(blocks), dim3(256), 0, stream, a);
    else if (a.dtype == 0 && a.head_dim == 64)
      hipLaunchKernelGGL((merge_kernel<64, float>), dim3(blocks), dim3(256), 0, stream, a);
    else
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

int32_t accept_chunks(int32_t rows, int32_t vocab) {
  const int32_t max_chunks = vocab / (256 * 8 * 4) > 1 ? vocab / (256 * 8 * 4) : 1;
  int32_t c = rows > 0 ? (2048 + rows - 1) / rows : 1;
  if (c > max_chunks) c = max_chunks;
  return c < 1 ? 1 : c;
}

hipError_t launch_accept(const AcceptArgs& a, hipStream_t stream) {
  const int rows = a.n_verify * (a.k_drafts + 1);
  if (rows == 0) return hipSuccess;
  if (a.logits_dtype == 1)
    hipLaunchKernelGGL(argmax_chunks<uint16_t>, dim3(rows * a.chunks), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(argmax_chunks<float>, dim3(rows * a.chunks), dim3(256), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(accept_kernel, dim3(a.n_verify), dim3(64), (a.k_drafts + 1) * sizeof(int), stream, a);
  return hipGetLastError();
}

hipError_t launch_kv_write(int32_t dtype, int32_t hkv, int32_t head_dim, int32_t block_size,
                           int64_t num_slots, void* k_cache, void* v_cache, const int64_t* slots,
                           const void* k_new, const void* v_new, int32_t n, int32_t* bad_slots,
                           hipStream_t stream) {
  if (n == 0) return hipSuccess;
  const int vec = dtype == 1 ? 8 : 4;
  const int64_t total = static_cast<int64_t>(n) * hkv * (head_dim / vec);
  const dim3 grid(static_cast<unsigned>((total + 255) / 256));
  if (dtype == 1)
    hipLaunchKernelGGL(kv_write_kernel<uint16_t>, grid, dim3(256), 0, stream, hkv, head_dim, block_size, num_slots,
                       static_cast<uint16_t*>(k_cache), static_cast<uint16_t*>(v_cache), slots,
                       static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new), n, bad_slots);
  else
    hipLaunchKernelGGL(kv_write_kernel<float>, grid, dim3(256), 0, stream, hkv, head_dim, block_size, num_slots,
                       static_cast<float*>(k_cache), static_cast<float*>(v_cache), slots,
                       static_cast<const float*>(k_new), static_cast<const float*>(v_new), n, bad_slots);
  return hipGetLastError();
}

hipError_t launch_kv_copy(int32_t dtype, int32_t hkv, int32_t head_dim, int32_t block_size,
                          void* k_cache, void* v_cache, int32_t src, int32_t dst, int32_t n_valid,
                          hipStream_t stream) {
  if (n_valid == 0) return hipSuccess;
  const int64_t total = static_cast<int64_t>(hkv) * n_valid * head_dim;
  const dim3 grid(static_cast<unsigned>((total + 255) / 256));
  if (dtype == 1)
    hipLaunchKernelGGL(kv_copy_kernel<uint16_t>, grid, dim3(256), 0, stream, hkv, head_dim, block_size,
                       static_cast<uint16_t*>(k_cache), static_cast<uint16_t*>(v_cache), src, dst, n_valid);
  else
    hipLaunchKernelGGL(kv_copy_kernel<float>, grid, dim3(256), 0, stream, hkv, head_dim, block_size,
                       static_cast<float*>(k_cache), static_cast<float*>(v_cache), src, dst, n_valid);
  return hipGetLastError();
}

}  // namespace spork
