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
#include <type_traits>

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
// bf16 partial attention. One workgroup of 4 waves owns a token range of one
// work item and up to 4*RTW 16-row tiles of its query rows; wave w computes
// tiles w, w+4, ... . The 32-token K/V tiles ("stages", 16 KB) are fetched
// once per workgroup: every thread issues 4 coalesced 16-byte loads per stage,
// kept NSTAGE_REGS stages ahead in registers, then written to one of two LDS
// slots and shared by all waves (one barrier per stage).
//
// LDS slot layout (1024 chunks of 16 bytes, XOR-swizzled so that the MFMA
// operand reads of each 8-lane group hit 8 different 128-byte bank groups):
//   K: chunk t*16 + (c ^ fk(t)) holds channels 8c..8c+7 of tile token t,
//      fk(t) = (t & 3) | ((t >> 1) & 4);
//   V: chunk 512 + d*4 + (q ^ ((d >> 1) & 3)) holds tokens 8q..8q+7 of
//      channel d (from the channel-major V blocks).
//
// Per stage and row tile (r16 = lane % 16, g = lane / 16 within the wave):
//   S^T = K Q^T via v_mfma_f32_16x16x32_bf16; A-row r16 of half hh is tile
//   token 8*(r16/4) + 4*hh + r16%4, so the lane receives scores of query row
//   r16 for tokens 8g + j (j = 0..7, halves concatenated); the contraction
//   slot of channel d is (k-step d/32, lane group (d%32)/8, element d%8) on
//   both operands.
//   O^T += V^T P^T: A = V^T (channel 16*dt + r16, tokens 8g..8g+7), B = the
//   lane's own 8 probabilities; the accumulator holds query row r16 at
//   channels 16*dt + 4g + i, so the rescale by the row's factor is lane-local.
// --------------------------------------------------------------------------
constexpr int kWgWaves = 4;
constexpr int kStageChunks = 1024;  // 32 tokens x (K + V) x 128 channels x 2 bytes / 16
constexpr int kStageRegs = 3;       // stages in flight in registers

__device__ __forceinline__ int k_swz(int t) { return (t & 3) | ((t >> 1) & 4); }

struct StageRegs {
  uint4 k0, k1, v0, v1;
};

// Zero the bf16 lanes of an 8-token chunk starting at position `first` whose
// position is at or past `end` (two tokens per 32-bit word).
__device__ __forceinline__ uint4 zero_past(uint4 v, int first, int end) {
  uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t lo = first + 2 * i < end ? 0x0000FFFFu : 0u;
    const uint32_t hi = first + 2 * i + 1 < end ? 0xFFFF0000u : 0u;
    w[i] &= lo | hi;
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}
__device__ __forceinline__ int v_swz(int d) { return (d >> 1) & 3; }

template <int RTW, int BS>
__global__ void __launch_bounds__(256, 2) attn_bf16(AttnArgs a) {
  constexpr int D = 128;
  static_assert(BS == 16 || BS == 32, "unsupported block size");
  __shared__ uint4 smem[2][kStageChunks];
  const WaveDesc w = a.waves[blockIdx.x];
  if (w.item < 0) return;
  const ItemDesc it = a.items[w.item];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const uint16_t* __restrict__ qg = static_cast<const uint16_t*>(a.q);
  const uint4* __restrict__ kc = static_cast<const uint4*>(a.k_cache);
  const uint4* __restrict__ vc = static_cast<const uint4*>(a.v_cache);
  const int32_t* __restrict__ table = a.tables + it.table_off;
  const int nb = it.n_blocks;
  const size_t head = static_cast<size_t>(it.kv_head);
  const size_t hkv = static_cast<size_t>(a.hkv);
  const int ntiles = (w.nrows + 15) >> 4;

  // Query operands and row horizons of this wave's tiles.
  bf16x8 qop[RTW][4];
  int hz[RTW];
  bool own[RTW];
#pragma unroll
  for (int j = 0; j < RTW; ++j) {
    const int tile = wave + kWgWaves * j;
    own[j] = tile < ntiles;
    const int i = tile * 16 + r16;
    if (own[j] && i < w.nrows) {
      const RowDesc rd = a.rows[it.row_off + w.row0 + i];
      hz[j] = rd.horizon;
      const uint4* qp = reinterpret_cast<const uint4*>(qg + static_cast<size_t>(rd.qidx) * D);
#pragma unroll
      for (int s = 0; s < 4; ++s) qop[j][s] = as_bf16x8(qp[4 * s + g]);
    } else {
      hz[j] = INT_MAX;  // padding row: zero query, never written
#pragma unroll
      for (int s = 0; s < 4; ++s) qop[j][s] = as_bf16x8(make_uint4(0, 0, 0, 0));
    }
  }
  int hmin = INT_MAX;
#pragma unroll
  for (int j = 0; j < RTW; ++j) hmin = min(hmin, hz[j]);
  hmin = wave_min_int(hmin);

  float m[RTW], l[RTW];
  f32x4 o[RTW][8];
#pragma unroll
  for (int j = 0; j < RTW; ++j) {
    m[j] = kNegInf;
    l[j] = 0.0f;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[j][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  const int tb0 = w.tok_lo & ~(kTileTokens - 1);
  const int nstage = (w.tok_hi - tb0 + kTileTokens - 1) / kTileTokens;

  // This thread's 4 chunks of a stage: K chunks tid and tid + 256 (tile
  // tokens tid/16 and 16 + tid/16), V chunks tid and tid + 256 (channels
  // tid/4 and 64 + tid/4).
  const int kt0 = tid >> 4;
  const int kc0 = (tid & 15) ^ k_swz(kt0);
  const int kc1 = (tid & 15) ^ k_swz(kt0 + 16);
  const int vd0 = tid >> 2;
  const int vq0 = (tid & 3) ^ v_swz(vd0);
  const int vq1 = (tid & 3) ^ v_swz(vd0 + 64);
  // Stages past the end reload the last stage (never stored): the loads stay
  // unconditional, which keeps the register pipeline straight-line.
  auto load_stage = [&](int st) __attribute__((always_inline)) {
    StageRegs r;
    const int tb = tb0 + min(st, nstage - 1) * kTileTokens;
    int bi0 = tb / BS, bi1 = (tb + 16) / BS;
    bi0 = bi0 < nb ? bi0 : nb - 1;
    bi1 = bi1 < nb ? bi1 : nb - 1;
    const size_t b0 = static_cast<size_t>(table[bi0]);
    const size_t b1 = static_cast<size_t>(table[bi1]);
    // K rows: token tb + t lives in block (t < 16 ? b0 : b1) at offset (tb + t) % BS
    r.k0 = kc[((b0 * hkv + head) * BS + (tb + kt0) % BS) * (D / 8) + kc0];
    r.k1 = kc[((b1 * hkv + head) * BS + (tb + 16 + kt0) % BS) * (D / 8) + kc1];
    // V^T rows: tokens tb + 8q .. +7 live in block (q < 2 ? b0 : b1)
    const size_t bv0 = vq0 < 2 ? b0 : b1;
    const size_t bv1 = vq1 < 2 ? b0 : b1;
    r.v0 = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(vc) +
                                           ((bv0 * hkv + head) * D + vd0) * BS + (tb + 8 * vq0) % BS);
    r.v1 = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(vc) +
                                           ((bv1 * hkv + head) * D + vd0 + 64) * BS + (tb + 8 * vq1) % BS);
    return r;
  };
  auto store_stage = [&](int st, StageRegs r) __attribute__((always_inline)) {
    const int tb = tb0 + st * kTileTokens;
    if (tb + kTileTokens > w.tok_hi) {
      // zero V of positions past the range: they may hold anything
      r.v0 = zero_past(r.v0, tb + 8 * vq0, w.tok_hi);
      r.v1 = zero_past(r.v1, tb + 8 * vq1, w.tok_hi);
    }
    uint4* slot = smem[st & 1];
    slot[tid] = r.k0;
    slot[tid + 256] = r.k1;
    slot[512 + tid] = r.v0;
    slot[512 + tid + 256] = r.v1;
  };

  // Tiles this wave owns: the first `nown` of its RTW slots (wave-uniform).
  int nown = 0;
#pragma unroll
  for (int j = 0; j < RTW; ++j) nown += own[j] ? 1 : 0;

  const float c = a.scale_log2;
  auto compute_tiles = [&](auto nown_c, int st) __attribute__((always_inline)) {
    constexpr int NT = decltype(nown_c)::value;
    const int tb = tb0 + st * kTileTokens;
    const uint4* slot = smem[st & 1];
    const bool edge = tb < w.tok_lo || tb + kTileTokens > w.tok_hi || tb + kTileTokens - 1 > hmin;
    f32x4 sc[NT][2];
#pragma unroll
    for (int j = 0; j < NT; ++j) sc[j][0] = sc[j][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int t = 8 * (r16 >> 2) + 4 * hh + (r16 & 3);
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const bf16x8 kop = as_bf16x8(slot[t * 16 + ((4 * s + g) ^ k_swz(t))]);
#pragma unroll
        for (int j = 0; j < NT; ++j)
          sc[j][hh] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop, qop[j][s], sc[j][hh], 0, 0, 0);
      }
    }
    bf16x8 pop[NT];
    float alpha[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      float sv[8] = {sc[j][0][0] * c, sc[j][0][1] * c, sc[j][0][2] * c, sc[j][0][3] * c,
                     sc[j][1][0] * c, sc[j][1][1] * c, sc[j][1][2] * c, sc[j][1][3] * c};
      if (edge) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int tk = tb + 8 * g + e;
          if (tk < w.tok_lo || tk >= w.tok_hi || tk > hz[j]) sv[e] = kNegInf;
        }
      }
      alpha[j] = softmax_step(sv, m[j], l[j]);
#pragma unroll
      for (int e = 0; e < 8; ++e) pop[j][e] = static_cast<__bf16>(sv[e]);
    }
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      const int d = 16 * dt + r16;
      const bf16x8 vop = as_bf16x8(slot[512 + d * 4 + (g ^ v_swz(d))]);
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        o[j][dt] *= alpha[j];
        o[j][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vop, pop[j], o[j][dt], 0, 0, 0);
      }
    }
  };
  auto compute_stage = [&](int st) __attribute__((always_inline)) {
    if (RTW >= 2 && nown == 2) compute_tiles(std::integral_constant<int, (RTW >= 2 ? 2 : 1)>{}, st);
    else if (nown == 1) compute_tiles(std::integral_constant<int, 1>{}, st);
  };

  // Software pipeline: stages st+1 .. st+kStageRegs-1 stay in flight while
  // stage st is written to LDS and computed.
  StageRegs ra = load_stage(0);
  StageRegs rb = load_stage(1);
  for (int st = 0; st < nstage; st += kStageRegs) {
    StageRegs rc = load_stage(st + 2);
    store_stage(st, ra);
    __syncthreads();
    compute_stage(st);
    if (st + 1 >= nstage) break;
    ra = load_stage(st + 3);
    store_stage(st + 1, rb);
    __syncthreads();
    compute_stage(st + 1);
    if (st + 2 >= nstage) break;
    rb = load_stage(st + 4);
    store_stage(st + 2, rc);
    __syncthreads();
    compute_stage(st + 2);
  }

#pragma unroll
  for (int j = 0; j < RTW; ++j) {
    if (!own[j]) continue;
    float lt = l[j] + __shfl_xor(l[j], 16);
    lt += __shfl_xor(lt, 32);
    const int i = (wave + kWgWaves * j) * 16 + r16;
    if (i < w.nrows) {
      const size_t pr = static_cast<size_t>(w.partial + i);
      if (g == 0) {
        a.part_ml[2 * pr] = m[j];
        a.part_ml[2 * pr + 1] = lt;
      }
#pragma unroll
      for (int dt = 0; dt < 8; ++dt)
        *reinterpret_cast<f32x4*>(a.part_o + pr * D + 16 * dt + 4 * g) = o[j][dt];
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

template <int BS>
AttnKernel pick_bf16(int row_tiles) {
  switch ((row_tiles + kWgWaves - 1) / kWgWaves) {
    case 1: return attn_bf16<1, BS>;
    case 2: return attn_bf16<2, BS>;
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
    if (bs == 16) return pick_bf16<16>(rt);
    if (bs == 32) return pick_bf16<32>(rt);
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

hipError_t launch_attn_partial(const AttnArgs& a, hipStream_t stream) {
  AttnKernel k = pick_attention(a.dtype, a.head_dim, a.block_size, a.row_tiles);
  if (k == nullptr) return hipErrorInvalidValue;
  const int threads = a.dtype == 1 ? 64 * kWgWaves : 64;
  if (a.n_waves > 0) hipLaunchKernelGGL(k, dim3(a.n_waves), dim3(threads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_merge(const AttnArgs& a, hipStream_t stream) {
  const int blocks = (a.n_out + 3) / 4;
  if (blocks == 0) return hipSuccess;
  if (a.dtype == 1 && a.head_dim == 128)
    hipLaunchKernelGGL((merge_kernel<128, __bf16>), dim3(blocks), dim3(256), 0, stream, a);
  else if (a.dtype == 0 && a.head_dim == 128)
    hipLaunchKernelGGL((merge_kernel<128, float>), dim3(blocks), dim3(256), 0, stream, a);
  else if (a.dtype == 0 && a.head_dim == 64)
    hipLaunchKernelGGL((merge_kernel<64, float>), dim3(blocks), dim3(256), 0, stream, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

int32_t accept_chunks(int32_t rows, int32_t vocab) {
  const int32_t max_chunks = vocab / (256 * 8 * 4) > 1 ? vocab / (256 * 8 * 4) : 1;
  int32_t c = rows > 0 ? (2048 + rows - 1) / rows : 1;
  if (c > max_chunks) c = max_chunks;
  return c < 1 ? 1 : c;
}

hipError_t launch_argmax(const AcceptArgs& a, hipStream_t stream) {
  const int rows = a.n_verify * (a.k_drafts + 1);
  if (rows == 0) return hipSuccess;
  if (a.logits_dtype == 1)
    hipLaunchKernelGGL(argmax_chunks<uint16_t>, dim3(rows * a.chunks), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(argmax_chunks<float>, dim3(rows * a.chunks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_accept_tail(const AcceptArgs& a, hipStream_t stream) {
  if (a.n_verify == 0) return hipSuccess;
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
