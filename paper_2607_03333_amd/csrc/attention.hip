// gfx950 (MI355X, CDNA4) attention kernels of the forked-decode hot path.
//
//  * attn_bf16 / attn_f32: partial attention of one work item's token range
//    for up to RT 16-row tiles of query rows (split-K). A work item is either
//    a fork group's shared prefix, read once for every member's rows
//    (Section 4.1: probes reuse the main thread's prefix KV), or one
//    thread's private range, where verify rows apply the causal rule over
//    the drafts (Section 4.3). Q.K^T and P.V run on MFMA with fp32
//    accumulation. bf16: K and V stream from HBM with 16-byte direct-to-LDS
//    loads (non-temporal) into a ring of LDS stages that the waves of a
//    workgroup share; fp32: 16-byte loads straight into registers.
//  * merge: log-sum-exp merge of an output row's partials (the batch's
//    maximum and weighted sum by DPP reductions over eight lanes), written
//    in the input dtype, plus the row's lse; the same launch runs the accept
//    of a verify step (Section 4.3, steps 2-3) and clears the persistent
//    launch's cursors for the next call.
#include "device_common.h"

namespace spork {
namespace {

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

// --------------------------------------------------------------------------
// bf16 partial attention. A persistent workgroup of NW waves (4, two per
// compute unit; or 8, one per compute unit) works through its list of units;
// a unit is a token range of one work item and up to NW*RTW 16-row tiles of
// its query rows; wave w computes tiles c, c + NW, ... (c = w, or w + 2 mod 4
// in the second 4-wave workgroup of a compute unit). The range streams through
// a ring of kRing LDS slots, one 32-token K/V tile ("stage", 16 KB) each,
// filled by direct global-to-LDS 16-byte loads (global_load_lds_dwordx4: lane
// i of an instruction lands at the instruction's LDS base + 16*i), so the
// stages in flight hold no registers. Each wave issues 16/NW such loads per
// stage (the first half of the waves the K half, the others the V half); a
// barrier publishes the next stage (4 waves) or the next two (8 waves) to all
// waves and frees the slots read before it.
//
// LDS slot layout (1024 chunks of 16 bytes). Bank model (measured on
// gfx950): 64 banks of 4 bytes, so a 16-byte slot s sits in bank group
// s mod 16; a ds_read_b128 serves a wave in four groups of 16 lanes (half
// lane >> 5, phase = parity of lane bits 2-4: lanes 0-3, 12-15, 20-27 |
// 4-11, 16-19, 28-31 of each half), and inside a group distinct addresses
// in one bank group serialise. Both operand reads below are conflict-free:
//   K: chunk t*16 + (c ^ fk(t)) holds channels 8c..8c+7 of tile token t,
//      fk(t) = (t & 3) | ((t >> 1) & 12);
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
constexpr int kStageChunks = 1024;  // 32 tokens x (K + V) x 128 channels x 2 bytes / 16
// LDS stages per workgroup: 4 for two 4-wave workgroups on a compute unit, 8
// for one 8-wave workgroup. A barrier publishes two stages (4-wave: 2 in
// flight, 8-wave: 6). Against one stage per barrier this halves the barriers,
// and the waves drift apart inside a pair instead of all reading the same
// operands right after every barrier: K = 16 verify step 8-10% faster, K = 50
// verify 2-3%, probe prefill 1-2%, and on the 4-wave decode loop (with a
// stage fewer in flight) the Qwen3-4B batch 3.6% and the bench workload 1.6%
// (the fork tree 0.8% slower); four per barrier: slower. In the 8-wave loop
// the second stage of a pair is published with the first, so its K operands
// are read into registers behind the first stage's softmax and its score
// products start without an LDS round trip (K = 16 verify step 3% faster,
// K = 50 2%, probe prefill 1%).
template <int NW>
constexpr int ring_of() { return NW == 4 ? 4 : 8; }
constexpr int kPer = 2;  // stages a barrier publishes

// Wait until at most `after` (0..7) stages of this wave's direct-to-LDS
// loads (LPW per stage), and no older vector load, are still in flight.
template <int LPW>
__device__ __forceinline__ void wait_stage(int after);
// Cache-policy bits of the K/V loads: non-temporal. Every KV byte is read
// once per launch, and streaming loads marked this way reach 7.2 TB/s on
// MI355X against 5.9 TB/s with the default policy (measured with the
// direct-to-LDS read-ceiling kernel in the same ring shape).
constexpr int kNonTemporal = 2;
constexpr int kUnitBlocks = kUnitTableEntries;   // block-table entries a unit may span (see kMaxUnitTokens)
constexpr float kRescaleSlack = 8.0f;  // base-2 headroom before the reference max moves
constexpr float kRescaleSum = 256.0f;  // 2^kRescaleSlack: bound on a lane's 8 probabilities of a row

typedef __attribute__((address_space(3))) void* lds_void_ptr;
typedef __attribute__((address_space(1))) void* global_void_ptr;

__device__ __forceinline__ int k_swz(int t) { return (t & 3) | ((t >> 1) & 12); }
__device__ __forceinline__ int v_swz(int d) { return (d >> 1) & 3; }

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

// LDS operand reads outside the compiler's view. The compiler cannot tell the
// direct-to-LDS loads of later stages from these reads of the current stage
// and would otherwise wait for every load in flight before each read. The
// waits are explicit: lds_wait() takes the destination registers as in-out
// operands, so no consumer can be scheduled before it.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void_ptr)(const_cast<void*>(p))));
}

template <int OFF = 0>
__device__ __forceinline__ u32x4 lds_read_b128(uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset field");
  u32x4 r;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF) : "memory");
  return r;
}

// The block-table entries of one stage, read from LDS at a wave-uniform
// address without a wait: the two entries of the stage's halves (the staged
// table holds each 32-token block's entry twice, so both block sizes read one
// pair). tab_wait() waits for the read and takes the registers as in-out
// operands, so no use moves above it. The read's own output registers are the
// pair: any copy of a register the read has not yet written (say, building
// the pair from one 32-bit result) would copy stale contents, since the
// compiler does not know the read is still in flight.
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ u32x2 tab_read(uint32_t addr) {
  u32x2 r;
  asm volatile("ds_read_b64 %0, %1" : "=v"(r) : "v"(addr) : "memory");
  return r;
}
__device__ __forceinline__ void tab_wait(u32x2& r) { asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(r) : : "memory"); }
template <int N>
__device__ __forceinline__ void tab_wait_all(u32x2 (&r)[N]) {
#pragma unroll
  for (int i = 0; i < N; ++i) tab_wait(r[i]);
}

// Wait for all LDS reads but the 8 issued last (LDS reads complete in order).
__device__ __forceinline__ void lds_wait_but8(u32x4 (&r)[8]) {
  asm volatile("s_waitcnt lgkmcnt(8)"
               : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]), "+v"(r[4]), "+v"(r[5]), "+v"(r[6]),
                 "+v"(r[7])
               :
               : "memory");
}

template <int N>
__device__ __forceinline__ void lds_wait(u32x4 (&r)[N]) {
  static_assert(N == 8, "lds_wait expects 8 registers");
  asm volatile("s_waitcnt lgkmcnt(0)"
               : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]), "+v"(r[4]), "+v"(r[5]), "+v"(r[6]),
                 "+v"(r[7])
               :
               : "memory");
}

// Workgroup-uniform reads of a unit's descriptors from the plan image (which
// no kernel writes while the attention launch runs) as scalar loads, on the
// scalar cache and its own counter, instead of vector loads that queue behind
// the stream's loads. Exactly the descriptor's bytes are read.
typedef int32_t i32x2 __attribute__((ext_vector_type(2)));
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x8 __attribute__((ext_vector_type(8)));
__device__ __forceinline__ WaveDesc load_wave_desc(const WaveDesc* p) {
  static_assert(sizeof(WaveDesc) == 24, "WaveDesc layout");
  i32x4 x;
  i32x2 y;
  asm volatile("s_load_dwordx4 %0, %2, 0x0\n\ts_load_dwordx2 %1, %2, 0x10\n\ts_waitcnt lgkmcnt(0)"
               : "=s"(x), "=s"(y)
               : "s"(p)
               : "memory");
  return WaveDesc{x[0], x[1], x[2], x[3], y[0], y[1]};
}
__device__ __forceinline__ ItemDesc load_item_desc(const ItemDesc* p) {
  static_assert(sizeof(ItemDesc) == 32, "ItemDesc layout");
  i32x8 x;
  asm volatile("s_load_dwordx8 %0, %1, 0x0\n\ts_waitcnt lgkmcnt(0)" : "=s"(x) : "s"(p) : "memory");
  ItemDesc it;
  static_assert(sizeof(it) == sizeof(x), "ItemDesc layout");
  __builtin_memcpy(&it, &x, sizeof(it));
  return it;
}
__device__ __forceinline__ int load_int_uniform(const int32_t* p) {
  int x;
  asm volatile("s_load_dword %0, %1, 0x0\n\ts_waitcnt lgkmcnt(0)" : "=s"(x) : "s"(p) : "memory");
  return x;
}

// Workgroup barrier that publishes this wave's LDS writes (and no global
// memory operation: no fence).
__device__ __forceinline__ void barrier_lds() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Workgroup barrier without the memory fence of __syncthreads(): callers make
// their own direct-to-LDS loads complete first (wait_vmcnt). The memory
// clobber keeps loads, stores and LDS operations on their side of it.
__device__ __forceinline__ void barrier_nofence() { asm volatile("s_barrier" ::: "memory"); }

// s_waitcnt on the vector-memory counter only (expcnt and lgkmcnt left open).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

template <int LPW>
__device__ __forceinline__ void wait_stage(int after) {
  static_assert(7 * LPW < 64, "vmcnt range");
  switch (after) {
    case 7: wait_vmcnt<7 * LPW>(); break;
    case 6: wait_vmcnt<6 * LPW>(); break;
    case 5: wait_vmcnt<5 * LPW>(); break;
    case 4: wait_vmcnt<4 * LPW>(); break;
    case 3: wait_vmcnt<3 * LPW>(); break;
    case 2: wait_vmcnt<2 * LPW>(); break;
    case 1: wait_vmcnt<LPW>(); break;
    default: wait_vmcnt<0>(); break;
  }
}

template <int RTW, int BS, int NW>
__global__ void __launch_bounds__(64 * NW, (NW == 4 ? 2 : 1)) attn_bf16(AttnArgs a) {
  constexpr int D = 128;
  constexpr int kRing = ring_of<NW>();
  constexpr int LPW = 16 / NW;  // direct-to-LDS loads per wave per 16 KB stage
  constexpr int NT_ = 64 * NW;  // threads
  static_assert(BS == 16 || BS == 32, "unsupported block size");
  static_assert(NW == 4 || NW == 8, "workgroups of 4 or 8 waves");
  __shared__ uint4 smem[kRing][kStageChunks];
  __shared__ __align__(16) int tab[kUnitBlocks];
  __shared__ int next_unit;
  // Persistent workgroup: it takes the next unit of its compute unit's list
  // (shared with the other workgroup resident there) until the list is done.
  const int tid = threadIdx.x;
  const int list = static_cast<int>(blockIdx.x) % a.n_lists;
  const int list0 = load_int_uniform(a.wg_off + list), list_len = load_int_uniform(a.wg_off + list + 1) - list0;
  // Thread 0 takes each unit before the workgroup needs it: the first here,
  // each next one at the end of the current unit, before its partial results
  // are stored, so neither the atomic's round trip nor the stores' sit
  // between two units. A barrier without a memory fence publishes the take.
  if (tid == 0) next_unit = atomicAdd(a.cursors + list * kCursorStride, 1);
  for (;;) {
  barrier_lds();
  const int taken = __builtin_amdgcn_readfirstlane(next_unit);
  if (taken < 0 || taken >= list_len) break;
  const WaveDesc w = load_wave_desc(a.waves + list0 + taken);
  if (w.item < 0) {  // padding (not emitted on persistent lists): every wave reads next_unit first
    barrier_nofence();
    if (tid == 0) next_unit = atomicAdd(a.cursors + list * kCursorStride, 1);
    continue;
  }
  const ItemDesc it = load_item_desc(a.items + w.item);
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  // Row tiles go to waves by `cw`, the wave index rotated by two in the
  // second workgroup of a compute unit (workgroups b and b + n_lists share
  // one): wave w of both shares SIMD w, and with 5-7 tiles (two for some
  // waves, one for others) the rotation pairs each wave holding two tiles
  // with one holding one.
  const int cw = NW == 4 ? (wave + 2 * (static_cast<int>(blockIdx.x) / a.n_lists)) & 3 : wave;
  const int lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const uint16_t* __restrict__ qg = static_cast<const uint16_t*>(a.q);
  const uint16_t* __restrict__ kc = static_cast<const uint16_t*>(a.k_cache);
  const uint16_t* __restrict__ vc = static_cast<const uint16_t*>(a.v_cache);
  const int32_t* __restrict__ table = a.tables + it.table_off;
  // Tokens appended to a private range's thread since the plan was made: the
  // range's last unit, its rows' horizons and its table grow by them.
  const int grow = it.grow;
  const int tok_hi = w.tok_hi == it.hi ? w.tok_hi + grow : w.tok_hi;
  const int nb = grow != 0 ? (it.hi + grow + BS - 1) / BS : it.n_blocks;
  const size_t head = static_cast<size_t>(it.kv_head);
  const size_t hkv = static_cast<size_t>(a.hkv);
  const int ntiles = (w.nrows + 15) >> 4;

  const int tb0 = w.tok_lo & ~(kTileTokens - 1);
  const int nstage = (tok_hi - tb0 + kTileTokens - 1) / kTileTokens;

  // Row descriptors of this wave's tiles, loaded together with the unit's
  // block table (below); the query rows they name are loaded once the table
  // is staged, and complete behind the ring's first loads.
  RowDesc rdesc[RTW];
  bool own[RTW], has_row[RTW];
#pragma unroll
  for (int j = 0; j < RTW; ++j) {
    const int tile = cw + NW * j;
    own[j] = tile < ntiles;
    const int i = tile * 16 + r16;
    has_row[j] = own[j] && i < w.nrows;
    rdesc[j] = a.rows[it.row_off + w.row0 + (has_row[j] ? i : 0)];  // padding lanes: the unit's first row, unused
  }
  // The unit's slice of the block table, staged in LDS before the ring
  // starts and read per stage outside the compiler's view (a vector load of
  // the table inside the loop would make its wait also wait for every
  // direct-to-LDS load issued before it), one stage ahead of its use. Stage
  // st reads the pair at tab[2*st]: with 16-token blocks tab[i] = table entry
  // tb0/BS + i, with 32-token blocks tab[2i] = tab[2i + 1] = entry tb0/BS + i
  // (entries clamped to the table).
  constexpr int kDup = BS == 16 ? 1 : 2;
  const int tab0 = tb0 / BS;
  const int ntab = min((tb0 + nstage * kTileTokens + 16) / BS - tab0 + 1, kUnitBlocks / kDup);  // planner keeps it below
  for (int i = tid; i < ntab; i += NT_) {
    const int bi = tab0 + i;
    const int e = table[bi < nb ? bi : nb - 1];
#pragma unroll
    for (int d = 0; d < kDup; ++d) tab[kDup * i + d] = e;
  }

  // Query operands and row horizons of this wave's tiles. A padding lane
  // (past the slice's rows) computes on the unit's first row with no causal
  // limit and is never stored; loading it like the others keeps the query
  // loads free of branches, whose merges would wait for them here.
  bf16x8 qop[RTW][4];
  int hz[RTW];
#pragma unroll
  for (int j = 0; j < RTW; ++j) {
    hz[j] = has_row[j] ? rdesc[j].horizon + grow : INT_MAX;
    const uint4* qp = reinterpret_cast<const uint4*>(qg + static_cast<size_t>(rdesc[j].qidx) * D);
#pragma unroll
    for (int s = 0; s < 4; ++s) qop[j][s] = as_bf16x8(qp[4 * s + g]);
  }
  int hmin = INT_MAX;
#pragma unroll
  for (int j = 0; j < RTW; ++j) hmin = min(hmin, hz[j]);
  hmin = wave_min_int(hmin);
  int nown = 0;  // tiles this wave owns: the first `nown` of its RTW slots
#pragma unroll
  for (int j = 0; j < RTW; ++j) nown += own[j] ? 1 : 0;

  float m[RTW], l[RTW];
  f32x4 o[RTW][8];
#pragma unroll
  for (int j = 0; j < RTW; ++j) {
    m[j] = kNegInf;
    l[j] = 0.0f;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[j][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // This lane's 4 chunks of a stage: instruction k of wave w fills chunks
  // (4w + k)*64 + lane. Waves 0-1: K chunks (token t, channel group c);
  // waves 2-3: V chunks (channel d, token octet q). The element offset inside
  // a block and the block (first or second of the stage) are fixed per lane.
  size_t off[LPW];
  bool second[LPW];
#pragma unroll
  for (int k = 0; k < LPW; ++k) {
    const int chunk = (LPW * wave + k) * 64 + lane;
    if (wave < NW / 2) {
      const int t = chunk >> 4;
      const int cg = (chunk & 15) ^ k_swz(t);
      second[k] = BS == 16 && t >= 16;
      off[k] = static_cast<size_t>(t % BS) * D + 8 * cg;
    } else {
      const int d = (chunk - 512) >> 2;
      const int q = (chunk & 3) ^ v_swz(d);
      second[k] = BS == 16 && q >= 2;
      off[k] = static_cast<size_t>(d) * BS + (8 * q) % BS;
    }
  }
  const uint16_t* pool = wave < NW / 2 ? kc : vc;
  barrier_lds();  // the table is in LDS; the query loads may still be in flight
  // Table entries of stage `st` (clamped to the unit's last stage), read
  // without a wait.
  const uint32_t tab_base = lds_addr(&tab[0]);
  auto stage_entries = [&](int st) __attribute__((always_inline)) {
    const int s = min(st, nstage - 1);
    return tab_read(tab_base + 8u * static_cast<uint32_t>(s));
  };
  // Issue the direct-to-LDS loads of stage `st` into ring slot st % kRing,
  // `ent` holding its table entries (already waited for).
  auto issue_stage = [&](int st, const u32x2& ent) __attribute__((always_inline)) {
    const int e0 = __builtin_amdgcn_readfirstlane(static_cast<int>(ent.x));
    const int e1 = __builtin_amdgcn_readfirstlane(static_cast<int>(ent.y));
    const size_t base0 = (static_cast<size_t>(e0) * hkv + head) * (static_cast<size_t>(BS) * D);
    const size_t base1 = (static_cast<size_t>(e1) * hkv + head) * (static_cast<size_t>(BS) * D);
    uint4* slot = smem[st % kRing];
#pragma unroll
    for (int k = 0; k < LPW; ++k) {
      const uint16_t* src = pool + (second[k] ? base1 : base0) + off[k];
      __builtin_amdgcn_global_load_lds((global_void_ptr)src, (lds_void_ptr)(slot + (LPW * wave + k) * 64), 16, 0,
                                       kNonTemporal);
    }
  };

  // Per-lane LDS byte addresses of the MFMA operands inside ring slot 0
  // (slot k adds k * 16 KB as an immediate offset):
  //   K operand (half hh, k-step s): token t = 8*(r16/4) + 4*hh + r16%4,
  //     chunk t*16 + ((4s + g) ^ fk(t));
  //   V operand (channel tile dt): chunk 512 + 4*(16*dt + r16) + (g ^ ((r16 >> 1) & 3)),
  //     i.e. a per-lane base plus 1024 bytes per dt.
  //   The second half's token is the first half's plus 4 with the same
  //   swizzle, so its addresses are the first half's plus 1024 bytes.
  uint32_t kaddr[4];
  {
    const int t = 8 * (r16 >> 2) + (r16 & 3);
#pragma unroll
    for (int s = 0; s < 4; ++s) kaddr[s] = 16u * (t * 16 + ((4 * s + g) ^ k_swz(t)));
  }
  const uint32_t smem_base = lds_addr(&smem[0][0]);
  const uint32_t vaddr = smem_base + 16u * (512 + 4 * r16 + (g ^ ((r16 >> 1) & 3)));
#pragma unroll
  for (int i = 0; i < 4; ++i) kaddr[i] += smem_base;

  // Softmax in base 2 with a lazily moved reference max: scores enter as
  // p = 2^(s*c - m) with m the row's reference; m (and the accumulator, by
  // 2^(m_old - m_new)) moves only when a lane's probabilities of the row sum
  // past 2^kRescaleSlack, so p <= 2^kRescaleSlack and most stages skip the
  // rescale. The merge only needs (m, l, o) to be consistent, not m to be the
  // exact maximum.
  const float c = a.scale_log2;
  // One stage for NT owned tiles, reading ring slot (st % kRing).
  auto read_k = [&](u32x4 (&kr)[8], int st) __attribute__((always_inline)) {
    const uint32_t soff = static_cast<uint32_t>(st % kRing) * (kStageChunks * 16);
#pragma unroll
    for (int i = 0; i < 4; ++i) kr[i] = lds_read_b128(kaddr[i] + soff);
#pragma unroll
    for (int i = 0; i < 4; ++i) kr[4 + i] = lds_read_b128<1024>(kaddr[i] + soff);
  };
  // PRE: kr already holds this stage's K (read during the previous stage).
  // NEXT: read the next stage's K into kr behind this stage's softmax.
  auto compute_tiles = [&](auto nt_c, auto pre_c, auto next_c, int st, u32x4 (&kr)[8]) __attribute__((always_inline)) {
    constexpr int NT = decltype(nt_c)::value;
    constexpr bool PRE = decltype(pre_c)::value, NEXT = decltype(next_c)::value;
    const int tb = tb0 + st * kTileTokens;
    const uint32_t soff = static_cast<uint32_t>(st % kRing) * (kStageChunks * 16);
    const bool edge = tb < w.tok_lo || tb + kTileTokens > tok_hi || tb + kTileTokens - 1 > hmin;
    if constexpr (!PRE) read_k(kr, st);
    lds_wait(kr);
    f32x4 sc[NT][2];
#pragma unroll
    for (int j = 0; j < NT; ++j) sc[j][0] = sc[j][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int j = 0; j < NT; ++j)
          sc[j][hh] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kr[4 * hh + s]),
                                                               qop[j][s], sc[j][hh], 0, 0, 0);
    const uint32_t va = vaddr + soff;
    u32x4 vr[8];
    vr[0] = lds_read_b128<0 * 1024>(va);
    vr[1] = lds_read_b128<1 * 1024>(va);
    vr[2] = lds_read_b128<2 * 1024>(va);
    vr[3] = lds_read_b128<3 * 1024>(va);
    vr[4] = lds_read_b128<4 * 1024>(va);
    vr[5] = lds_read_b128<5 * 1024>(va);
    vr[6] = lds_read_b128<6 * 1024>(va);
    vr[7] = lds_read_b128<7 * 1024>(va);
    float sv[NT][8];
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int e = 0; e < 8; ++e) sv[j][e] = sc[j][e >> 2][e & 3];
    // Masking of positions outside the range or past a row's horizon (first
    // and last stages of a unit, causal rows).
    auto mask_tile = [&](int j) __attribute__((always_inline)) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int tk = tb + 8 * g + e;
        if (tk < w.tok_lo || tk >= tok_hi || tk > hz[j]) sv[j][e] = kNegInf;
      }
    };
    // Softmax of tile j: the lane's 8 probabilities of its row against the
    // row's reference. Common case: they sum to at most 2^kRescaleSlack
    // (which bounds each of them). Only when some lane of the wave sums past
    // that, or a row has no reference yet, are the row maxima reduced across
    // lanes, the reference moved where it lags by more than kRescaleSlack
    // (rows that did not trigger keep theirs) and the probabilities
    // recomputed.
    auto softmax_tile = [&](int j) __attribute__((always_inline)) {
      float ps = 0.0f;
      float pv[8];
      {
        const float mu = m[j] == kNegInf ? 0.0f : m[j];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          pv[e] = exp2_fast(__builtin_fmaf(sv[j][e], c, -mu));
          ps += pv[e];
        }
      }
      if constexpr (NW == 8) {
        // Scheduling hint for the block that holds the previous tile's P.V:
        // alternate one MFMA with three vector instructions of this tile's
        // exponentials instead of issuing the MFMAs back to back.
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
          __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);  // VALU
        }
      }
      if (__ballot(!(ps <= kRescaleSum) || m[j] == kNegInf) != 0) {
        float mx = fmaxf(fmaxf(fmaxf(sv[j][0], sv[j][1]), fmaxf(sv[j][2], sv[j][3])),
                         fmaxf(fmaxf(sv[j][4], sv[j][5]), fmaxf(sv[j][6], sv[j][7])));
        mx *= c;
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        if (mx > m[j] + kRescaleSlack) {  // row-uniform: all 4 lanes of the row agree
          const float alpha = exp2_fast(m[j] - mx);  // 0 for a row's first visible tile
          l[j] *= alpha;
#pragma unroll
          for (int dt = 0; dt < 8; ++dt) o[j][dt] *= alpha;
          m[j] = mx;
        }
        const float mu = m[j] == kNegInf ? 0.0f : m[j];
        ps = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          pv[e] = exp2_fast(__builtin_fmaf(sv[j][e], c, -mu));
          ps += pv[e];
        }
      }
      bf16x8 pop;
#pragma unroll
      for (int e = 0; e < 8; ++e) pop[e] = static_cast<__bf16>(pv[e]);
      l[j] += ps;
      return pop;
    };
    auto pv_tile = [&](int j, const bf16x8& pop) __attribute__((always_inline)) {
#pragma unroll
      for (int dt = 0; dt < 8; ++dt)
        o[j][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vr[dt]), pop, o[j][dt], 0, 0, 0);
    };
    // Positions past the range may hold anything: zero their V (0 * NaN
    // would poison the accumulator).
    auto zero_past_range = [&]() __attribute__((always_inline)) {
      if (tb + kTileTokens > tok_hi) {
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) {
          const uint4 z = zero_past(make_uint4(vr[dt][0], vr[dt][1], vr[dt][2], vr[dt][3]), tb + 8 * g, tok_hi);
          vr[dt] = u32x4{z.x, z.y, z.z, z.w};
        }
      }
    };
    if constexpr (NW == 8) {
      // One workgroup per compute unit, the multi-row (prefill, long verify)
      // shapes: the P.V of tile j - 1 is issued before the softmax of tile j,
      // so the matrix cores work on one tile while the vector ALUs take the
      // exponentials of the next.
      // One branch masks all tiles, so the tiles' arithmetic below stays in
      // one basic block.
      if (edge) {
#pragma unroll
        for (int j = 0; j < NT; ++j) mask_tile(j);
      }
      bf16x8 pop = softmax_tile(0);
      if constexpr (NEXT) {
        read_k(kr, st + 1);
        lds_wait_but8(vr);
      } else {
        lds_wait(vr);
      }
      zero_past_range();
#pragma unroll
      for (int j = 1; j < NT; ++j) {
        pv_tile(j - 1, pop);
        pop = softmax_tile(j);
      }
      pv_tile(NT - 1, pop);
    } else {
      // Two workgroups per compute unit: the other workgroup's waves fill the
      // matrix cores; all softmaxes first, then the P.V products.
      bf16x8 pop[NT];
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        if (edge) mask_tile(j);
        pop[j] = softmax_tile(j);
      }
      lds_wait(vr);
      zero_past_range();
#pragma unroll
      for (int dt = 0; dt < 8; ++dt)
#pragma unroll
        for (int j = 0; j < NT; ++j)
          o[j][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vr[dt]), pop[j], o[j][dt], 0,
                                                             0, 0);
    }
  };

  // Prologue: the first kAhead = kRing - 2 stages in flight. The query rows,
  // loaded before them, complete first (vector loads complete in order):
  // this wait leaves only the prologue's loads in flight, and no wait for the
  // query rows lands inside the loop.
  constexpr int kAhead = kRing - kPer;
#pragma unroll
  for (int st = 0; st < kAhead; ++st) {
    if (st < nstage) {
      u32x2 ent = stage_entries(st);
      tab_wait(ent);
      issue_stage(st, ent);
    }
  }
  wait_stage<LPW>(min(kAhead, nstage));

  // The ring loop, specialised on the number of tiles this wave owns so that
  // no branch on it sits inside the loop. Every wave runs nstage barriers.
  auto run = [&](auto nt_c) __attribute__((always_inline)) {
    constexpr int NT = decltype(nt_c)::value;
    // Every kPer stages: wait for this wave's loads of the next kPer stages
    // (the stages issued after them, at most kAhead - kPer, may stay in
    // flight), one barrier that makes them visible to all waves and frees
    // the slots of the previous kPer stages, and the loads of kPer more
    // stages into those slots. The table entries of the stages a barrier
    // issues are read one barrier ahead: the operand waits of the compute in
    // between cover their latency.
    u32x2 ent[kPer];
#pragma unroll
    for (int q = 0; q < kPer; ++q) ent[q] = stage_entries(kAhead + q);
    u32x4 kr[8];
    for (int st = 0; st < nstage; st += kPer) {
      wait_stage<LPW>(max(0, min(kAhead - kPer, nstage - kPer - st)));
      barrier_nofence();
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        if (st + kAhead + q < nstage) {
          tab_wait(ent[q]);
          issue_stage(st + kAhead + q, ent[q]);
        }
      }
#pragma unroll
      for (int q = 0; q < kPer; ++q) ent[q] = stage_entries(st + kRing + q);
      if constexpr (NT > 0) {
        if constexpr (NW == 8) {
          compute_tiles(nt_c, std::false_type{}, std::true_type{}, st, kr);
          if (st + 1 < nstage) compute_tiles(nt_c, std::true_type{}, std::false_type{}, st + 1, kr);
        } else {  // the 4-wave compute reads each stage's K itself
          compute_tiles(nt_c, std::false_type{}, std::false_type{}, st, kr);
          if (st + 1 < nstage) compute_tiles(nt_c, std::false_type{}, std::false_type{}, st + 1, kr);
        }
      }
    }
    wait_vmcnt<0>();
    // The LDS reads issued by inline assembly are invisible to the compiler's
    // wait tracking: a K prefetch for a stage past the unit's end and the
    // table entries read one barrier ahead are still in flight here. Wait
    // for them with their registers as operands, so that no later value is
    // placed in those registers before the reads have written them.
    tab_wait_all(ent);
    if constexpr (NW == 8) lds_wait(kr);
    // Every wave has read this unit's take (the ring loop's barriers follow
    // it): take the next unit now.
    int nxt = 0;
    if (tid == 0) nxt = atomicAdd(a.cursors + list * kCursorStride, 1);
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      float lt = l[j] + __shfl_xor(l[j], 16);
      lt += __shfl_xor(lt, 32);
      const int i = (cw + NW * j) * 16 + r16;
      if (i < w.nrows) {
        const size_t pr = static_cast<size_t>(a.part_slot[w.partial + i]);
        if (g == 0) {
          a.part_ml[2 * pr] = m[j];
          a.part_ml[2 * pr + 1] = lt;
        }
        // bf16, in register order: the lane's 32 channels 16*dt + 4*g + i
        // (dt = 0..7, i = 0..3) at row positions 32*g + 4*dt + i, four
        // 16-byte stores.
        u32x4* dst = reinterpret_cast<u32x4*>(static_cast<__bf16*>(a.part_o) + pr * D + 32 * g);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          bf16x8 h;
#pragma unroll
          for (int e = 0; e < 8; ++e) h[e] = static_cast<__bf16>(o[j][2 * q + (e >> 2)][e & 3]);
          dst[q] = __builtin_bit_cast(u32x4, h);
        }
      }
    }
    if (tid == 0) next_unit = nxt;
  };
  if (RTW >= 2 && nown == 2) run(std::integral_constant<int, (RTW >= 2 ? 2 : 1)>{});
  else if (nown == 1) run(std::integral_constant<int, 1>{});
  else run(std::integral_constant<int, 0>{});
  // The next take's barrier is reached by every wave only after its last
  // reads of this unit's ring slots, table and next_unit.
  }
  // Verify step: the greedy argmax over the logits fills the tail of the
  // launch. Workgroups whose lists are done take (row, chunk) units from one
  // shared cursor, so the compute units that finish early stream the logits
  // while the last attention units drain.
  if (a.tail_units > 0) {
    __syncthreads();  // every wave has read the last list take
    for (;;) {
      if (tid == 0) next_unit = atomicAdd(a.cursors + a.n_lists * kCursorStride, 1);
      __syncthreads();
      const int u = __builtin_amdgcn_readfirstlane(next_unit);
      if (u < 0 || u >= a.tail_units) break;
      const int row = u / a.acc.chunks, c = u % a.acc.chunks;
      uint64_t* key = a.acc.keys + static_cast<size_t>(row) * a.acc.chunks + c;
      const size_t roff = static_cast<size_t>(row) * a.acc.vocab;
      if (a.acc.logits_dtype == 1)
        argmax_unit<uint16_t, NT_, false>(static_cast<const uint16_t*>(a.acc.logits) + roff, a.acc.vocab,
                                          a.acc.chunks, c, key, nullptr);
      else
        argmax_unit<float, NT_, false>(static_cast<const float*>(a.acc.logits) + roff, a.acc.vocab, a.acc.chunks,
                                       c, key, nullptr);
      // The unit ends with thread 0 storing the key and the next take starts
      // with thread 0 taking a unit: this barrier keeps the two thread-0
      // regions apart, so the compiler cannot join them across the loop's
      // back edge into a loop whose waves run different barrier counts.
      __syncthreads();
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
  const int grow = it.grow;  // tokens appended since the plan (see the bf16 kernel)
  const int tok_hi = w.tok_hi == it.hi ? w.tok_hi + grow : w.tok_hi;
  const int nb = grow != 0 ? (it.hi + grow + BS - 1) / BS : it.n_blocks;
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
      hz[t] = rd.horizon + grow;
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
  for (int tb = w.tok_lo & ~(kTileTokens - 1); tb < tok_hi; tb += kTileTokens) {
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
        if (tb + kTileTokens > tok_hi) {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (tb + 16 * hh + 4 * g + i >= tok_hi) v[i] = 0.0f;
        }
        vop[hh][dt] = v;
      }
    }
    const bool edge = tb < w.tok_lo || tb + kTileTokens > tok_hi || tb + kTileTokens - 1 > hmin;
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
              if (tk < w.tok_lo || tk >= tok_hi || tk > hz[t]) sv[4 * hh + i] = kNegInf;
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
        const size_t pr = static_cast<size_t>(a.part_slot[w.partial + i]);
        if (g == 0) {
          a.part_ml[2 * pr] = m[t];
          a.part_ml[2 * pr + 1] = lt;
        }
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          *reinterpret_cast<f32x4*>(static_cast<float*>(a.part_o) + pr * D + 16 * dt + 4 * g) = o[t][dt];
      }
    }
  }
}

// --------------------------------------------------------------------------
// Log-sum-exp merge: one wave per output (query row x query head).
//   M = max m_i, L = sum 2^(m_i - M) l_i, O = sum 2^(m_i - M) o_i / L,
//   lse = (M + log2 L) ln 2. Partials with nothing visible (m = -inf, l = 0)
//   add nothing.
// Partials go in batches of 4 (outputs with at most 4) or 8. An output's
// partials are consecutive rows; lane i loads the (m, l) pair of partial i
// and every lane its channels of all the batch's rows, in one round trip.
// The batch maximum and the weighted sum of l are DPP reductions over lanes
// 0-7; unused slots repeat a valid row with weight 0. Batches after the
// first rescale the running sums to the new maximum.
// --------------------------------------------------------------------------
// Partial rows are in the input dtype: fp32 rows in channel order, bf16 rows
// (D = 128) in the bf16 attention writer's register order, channel
// 16*dt + 4*g + i at position 32*g + 4*dt + i. Lane `lane` reads positions
// PER*lane .. PER*lane + PER - 1 of every partial row (one coalesced pass
// over the row) and merges the channels stored there: channel PER*lane + e
// (fp32), or, for bf16, the pair merge_channel() + e (g = lane / 16,
// dt = lane / 2 mod 8, i = 2 * (lane mod 2) and i + 1).
template <int D, typename PT>
__device__ __forceinline__ int merge_channel(int lane) {
  if constexpr (std::is_same<PT, float>::value) {
    return lane * (D / 64);
  } else {
    static_assert(D == 128, "bf16 partial rows are 128 channels");
    return 16 * ((lane >> 1) & 7) + 4 * (lane >> 4) + 2 * (lane & 1);
  }
}

template <int D, typename PT>
__device__ __forceinline__ void load_partial(const AttnArgs& a, size_t row, int lane, float (&po)[D / 64]) {
  constexpr int PER = D / 64;
  if constexpr (std::is_same<PT, float>::value) {
    const float* src = static_cast<const float*>(a.part_o) + row * D + lane * PER;
#pragma unroll
    for (int e = 0; e < PER; ++e) po[e] = src[e];
  } else {
    const uint32_t w = reinterpret_cast<const uint32_t*>(static_cast<const __bf16*>(a.part_o) + row * D)[lane];
    po[0] = __uint_as_float(w << 16);
    po[1] = __uint_as_float(w & 0xFFFF0000u);
  }
}

// One batch of at most B partials (entries c0 .. c0 + k - 1 of the output's
// list), folded into the running (max, sum, accumulator).
template <int B, int D, typename PT>
__device__ __forceinline__ void merge_batch(const AttnArgs& a, int c0, int k, bool first, int lane, float& run_max,
                                            float& mu, float& sum, float (&acc)[D / 64]) {
  constexpr int PER = D / 64;
  // the output's partials are consecutive: rows c0 .. c0 + k - 1
  const float2 ml = reinterpret_cast<const float2*>(a.part_ml)[c0 + min(lane, k - 1)];
  float po[B][PER];
#pragma unroll
  for (int i = 0; i < B; ++i) load_partial<D, PT>(a, static_cast<size_t>(c0 + min(i, k - 1)), lane, po[i]);
  const bool live = lane < k;
  const float pm = live ? ml.x : kNegInf;
  const float pl = live ? ml.y : 0.0f;
  const float bm = lanes8_max(pm);  // lanes k.. hold -inf
  const float new_max = fmaxf(run_max, bm);
  const float new_mu = new_max == kNegInf ? 0.0f : new_max;
  if (!first) {
    const float alpha = exp2_fast(mu - new_mu);
    sum *= alpha;
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] *= alpha;
  }
  run_max = new_max;
  mu = new_mu;
  const float w = exp2_fast(pm - mu);  // lane i: weight of partial i, 0 for unused slots (pm = -inf)
  sum += lanes8_sum(w * pl);
#pragma unroll
  for (int i = 0; i < B; ++i) {
    const float wgt = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, w), i));
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] += wgt * po[i][e];
  }
}

template <int D, typename OutT>
__global__ void __launch_bounds__(256) merge_kernel(AttnArgs a) {
  constexpr int PER = D / 64;
  // The attention launch is done with its cursors: return them to zero for
  // the workspace's next call.
  if (blockIdx.x == 0)
    for (int i = threadIdx.x; i < a.n_cursors; i += 256) a.cursors[i * kCursorStride] = 0;
  const int merge_blocks = (a.n_out + 3) / 4;
  if (static_cast<int>(blockIdx.x) >= merge_blocks) {
    // fused accept: one verify thread per wave
    const int sv = (blockIdx.x - merge_blocks) * 4 + (threadIdx.x >> 6);
    if (sv < a.acc.n_verify) accept_unit(a.acc, sv);
    return;
  }
  const int o = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (o >= a.n_out) return;
  const int beg = a.merge_off[o], end = a.merge_off[o + 1];
  float acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.0f;
  float mu = 0.0f, sum = 0.0f, run_max = kNegInf;
  if (end - beg <= 4) {
    merge_batch<4, D, OutT>(a, beg, end - beg, true, lane, run_max, mu, sum, acc);
  } else {
    for (int c0 = beg; c0 < end; c0 += 8)
      merge_batch<8, D, OutT>(a, c0, min(8, end - c0), c0 == beg, lane, run_max, mu, sum, acc);
  }
  const float inv = sum > 0.0f ? 1.0f / sum : 0.0f;
  OutT* out = static_cast<OutT*>(a.out) + static_cast<size_t>(o) * D + merge_channel<D, OutT>(lane);
#pragma unroll
  for (int e = 0; e < PER; ++e) out[e] = static_cast<OutT>(acc[e] * inv);
  if (lane == 0 && a.lse != nullptr)
    a.lse[o] = sum > 0.0f ? (mu + __log2f(sum)) * kLn2 : kNegInf;
}

__global__ void __launch_bounds__(256) counter_reset_kernel(int32_t* counters, int32_t n) {
  for (int i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) counters[i] = 0;
}

// --------------------------------------------------------------------------
// Dispatch tables.
// --------------------------------------------------------------------------
typedef void (*AttnKernel)(AttnArgs);

template <int BS, int NW>
AttnKernel pick_bf16(int row_tiles) {
  switch ((row_tiles + NW - 1) / NW) {
    case 1: return attn_bf16<1, BS, NW>;
    case 2: return attn_bf16<2, BS, NW>;
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

// Exactly the shapes attention_supported (dispatch_rules.cpp) accepts.
AttnKernel pick_attention(int32_t dtype, int32_t d, int32_t bs, int32_t rt, int32_t waves) {
  if (dtype == 1 && d == 128 && (waves == 4 || waves == 8)) {
    if (bs == 16) return waves == 4 ? pick_bf16<16, 4>(rt) : pick_bf16<16, 8>(rt);
    if (bs == 32) return waves == 4 ? pick_bf16<32, 4>(rt) : pick_bf16<32, 8>(rt);
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

hipError_t launch_attn_partial(const AttnArgs& a, hipStream_t stream) {
  AttnKernel k = pick_attention(a.dtype, a.head_dim, a.block_size, a.row_tiles, a.wg_waves);
  if (k == nullptr) return hipErrorInvalidValue;
  const int threads = a.dtype == 1 ? 64 * a.wg_waves : 64;
  if (a.grid > 0) hipLaunchKernelGGL(k, dim3(a.grid), dim3(threads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_counter_reset(int32_t* counters, int32_t n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const int blocks = n / 256 + 1 < 64 ? n / 256 + 1 : 64;
  hipLaunchKernelGGL(counter_reset_kernel, dim3(blocks), dim3(256), 0, stream, counters, n);
  return hipGetLastError();
}

hipError_t launch_merge(const AttnArgs& a, hipStream_t stream) {
  int blocks = (a.n_out + 3) / 4 + (a.acc.n_verify + 3) / 4;
  if (blocks == 0 && a.n_cursors == 0) return hipSuccess;
  if (blocks == 0) blocks = 1;  // only the cursors to clear
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

}  // namespace spork
