// Kernel 3 of the fused BMU search: a shared-union super-tile.
//
// The union sweep of Section 4.1 reads each union row slice once per tile,
// so the rows that many tiles hold (the head of the feature law) are
// requested from L2 once per tile, and the tile size that keeps a wave's
// accumulators in VGPRs (T documents x K neurons per lane) caps the sharing.
// Here a workgroup of S waves takes a super-tile of D = S*T consecutive
// documents of the tiled order and one neuron slice of 64*K neurons: the
// super-tile's union (its own plan, D-bit membership masks) is swept once,
// each row slice fetched once per workgroup (one 1 KB row per wave
// instruction, 16 bytes per lane) straight into LDS, and every wave adds
// from LDS the rows that its own T documents hold.  Wave w owns documents
// w*T .. w*T+T-1 of the super-tile and their T x K accumulators, exactly as a
// kernel-1 wave owns a tile; its T-bit slice of each entry's mask drives the
// same wave-uniform dispatch, and its documents' dot products are summed in
// ascending feature order, so the results are bit-identical to kernel 1's.
//
// Pipeline: the union is cut into stages of P entries held in a ring of
// NSLOT LDS slots.  Each wave moves its P/S rows of a stage, and its own
// T-bit mask word of each of the stage's entries, with direct global-to-LDS
// loads (no registers), NSLOT-1 stages ahead of the adds.  Before stage s is
// added, each wave waits until its own loads of stage s have landed (a
// vector-memory count: the loads of the later stages may stay in flight),
// then one barrier makes every wave's part visible and closes stage s-1,
// whose slot the loads of stage s+NSLOT-1 then reuse.  The feature ids of
// those loads arrive with stage s itself (spare lanes of its mask load).
// Entries past the union's end load row 0 and get empty masks.  A wave adds
// only the entries of a stage its documents hold, in one of the dispatch
// forms of StDispatch below: row-major (a ballot over the stage's entry
// masks gives the needed rows, visited in ascending order with the next
// row's LDS read issued before the current row's adds) or document-major
// (per document, the stage entries it holds, from 16-bit document words that
// the plan stores per stage and the wave reads with scalar loads a stage
// ahead; for fp32 rows the whole stage's adds are one inline-assembly
// statement, and the last stage is peeled off the loop).
//
// Rotated sweep (the default document-major form): each super-tile starts its union
// at a stage chosen from its place in its XCD's work and wraps round, so that
// the super-tiles an XCD runs at once sweep the same part of the feature
// range at the same time and share their rows in that XCD's L2 (in ascending
// order they start at staggered times and spread over the whole range).  A
// document's dot product is then summed in that rotated order: a fixed order
// for a given plan and device, different from the ascending one in rounding.
//
// Included by the translation units that instantiate it; internal linkage.
#pragma once

#include "search_k1.h"

namespace som {
namespace {

typedef __attribute__((address_space(3))) void* lds_ptr;

// Byte offset of a __shared__ object in the workgroup's LDS.
__device__ __forceinline__ uint32_t lds_offset(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_ptr)(const_cast<void*>(p))));
}

// Direct global-to-LDS loads: lane i's 16 (or 4) bytes at `src` land at LDS
// byte m0 + 16*i (or 4*i); `m0` must be wave-uniform.  The loads count in the
// vector-memory counter like any load and write LDS when they return.  They
// are issued by inline assembly so that the compiler's own wait insertion
// (which cannot tell ring slots apart) does not drain them at every LDS
// read; the kernel waits for them itself (vm_wait) before its barriers.
__device__ __forceinline__ void dma_b128(const void* src, uint32_t m0) {
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "{m0}"(m0) : "memory");
}
__device__ __forceinline__ void dma_b32(const void* src, uint32_t m0) {
  asm volatile("s_nop 0\n\tglobal_load_lds_dword %0, off" ::"v"(src), "{m0}"(m0) : "memory");
}

// Wait until at most N vector-memory operations of this wave are in flight.
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Wait until at most `n` of this wave's stages are still in flight (OPS
// loads per stage); n is wave-uniform and at most NSLOT - 2.
template <int OPS, int NSLOT>
__device__ __forceinline__ void wait_stages(int n) {
  static_assert(NSLOT >= 2 && NSLOT <= 6 && (NSLOT - 2) * OPS < 64, "ring depth");
  if (NSLOT > 5 && n >= 4) return vm_wait<(NSLOT > 5 ? 4 : 0) * OPS>();
  if (NSLOT > 4 && n >= 3) return vm_wait<(NSLOT > 4 ? 3 : 0) * OPS>();
  if (NSLOT > 3 && n >= 2) return vm_wait<(NSLOT > 3 ? 2 : 0) * OPS>();
  if (NSLOT > 2 && n >= 1) return vm_wait<(NSLOT > 2 ? 1 : 0) * OPS>();
  vm_wait<0>();
}

__device__ __forceinline__ void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }

// The adds of a stage for a wave's eight documents, fp32 rows,
// document-major dispatch: w[j] holds the stage words of documents 2j (low
// half) and 2j + 1 (high half); for each set bit r of a document's word, in
// ascending order, the lane's 16 bytes of row r of the stage's LDS slot (at
// byte vbase + 1024 r) are added to that document's four accumulators.  One
// inline-assembly statement keeps the loop at three scalar instructions per
// row and each document's test at one: the compiler's form compares each
// cleared word with zero again after the s_and that has already set SCC,
// tests a half-word in two instructions, and pads every statement boundary
// with a wait state.  The row lands in v60-v63, which the statement clobbers.
#define SOM_DOC_ROWS(FIRST, D)                         \
  FIRST "\n\t"                                         \
  "s_cbranch_scc0 7f\n"                                 \
  "9:\n\t"                                             \
  "s_ff1_i32_b32 %[r], %[dm]\n\t"                      \
  "v_lshl_add_u32 %[va], %[r], 10, %[vb]\n\t"          \
  "ds_read_b128 v[60:63], %[va]\n\t"                   \
  "s_add_i32 %[r], %[dm], -1\n\t"                      \
  "s_and_b32 %[dm], %[dm], %[r]\n\t"                   \
  "s_waitcnt lgkmcnt(0)\n\t"                           \
  "v_add_f32_e32 %[" #D "0], v60, %[" #D "0]\n\t"      \
  "v_add_f32_e32 %[" #D "1], v61, %[" #D "1]\n\t"      \
  "v_add_f32_e32 %[" #D "2], v62, %[" #D "2]\n\t"      \
  "v_add_f32_e32 %[" #D "3], v63, %[" #D "3]\n\t"      \
  "s_cbranch_scc1 9b\n"                                \
  "7:\n\t"
#define SOM_DOC_ACC(D, A) [D##0] "+v"(A[0]), [D##1] "+v"(A[1]), [D##2] "+v"(A[2]), [D##3] "+v"(A[3])
__device__ __forceinline__ void add_stage_8docs_f32(float (&acc)[8][4], const uint32_t (&w)[4], uint32_t vbase) {
  uint32_t dm, r, va;
  asm volatile(SOM_DOC_ROWS("s_and_b32 %[dm], %[w0], 0xffff", a) SOM_DOC_ROWS("s_lshr_b32 %[dm], %[w0], 16", b)
               SOM_DOC_ROWS("s_and_b32 %[dm], %[w1], 0xffff", c) SOM_DOC_ROWS("s_lshr_b32 %[dm], %[w1], 16", d)
               SOM_DOC_ROWS("s_and_b32 %[dm], %[w2], 0xffff", e) SOM_DOC_ROWS("s_lshr_b32 %[dm], %[w2], 16", f)
               SOM_DOC_ROWS("s_and_b32 %[dm], %[w3], 0xffff", g) SOM_DOC_ROWS("s_lshr_b32 %[dm], %[w3], 16", h)
               : SOM_DOC_ACC(a, acc[0]), SOM_DOC_ACC(b, acc[1]), SOM_DOC_ACC(c, acc[2]),
                 SOM_DOC_ACC(d, acc[3]), SOM_DOC_ACC(e, acc[4]), SOM_DOC_ACC(f, acc[5]),
                 SOM_DOC_ACC(g, acc[6]), SOM_DOC_ACC(h, acc[7]), [dm] "=&s"(dm), [r] "=&s"(r), [va] "=&v"(va)
               : [w0] "s"(w[0]), [w1] "s"(w[1]), [w2] "s"(w[2]), [w3] "s"(w[3]), [vb] "v"(vbase)
               : "v60", "v61", "v62", "v63", "scc", "memory");
}
#undef SOM_DOC_ACC
#undef SOM_DOC_ROWS

// Dispatch of a stage's rows to a wave's documents (both add every row in
// ascending feature order, so their results are bit-identical):
//   kStRowMajor: visit each entry some document of the wave holds (one
//     ballot over the stage's entry-major masks), read its row from LDS once,
//     then a scalar branch tree over the wave's documents (a test per group
//     of four, then one per document);
//   kStDocMajor: the plan stores each stage's masks document-major (one
//     16-bit word per document: the stage entries it holds); the wave's T
//     words arrive in scalar registers with one scalar load issued a stage
//     ahead, and per document each held entry is read from LDS and added,
//     with a static accumulator index and no per-row scalar branch tree;
//   kStDocRotated: kStDocMajor over the stages in rotated order (stage s0 to
//     the last, then stage 0 to s0 - 1; s0 from the super-tile's phase).
enum StDispatch { kStRowMajor = 0, kStDocMajor = 1, kStDocRotated = 2 };

template <typename WT, int T, int K, int S, int P, int NSLOT, int DISP>
__global__ void __launch_bounds__(S * 64)
k_search_st(SearchArgs a) {
  constexpr int E = Storage<WT>::kE;  // elements per 128-bit load
  static_assert(K == E, "one 128-bit load per lane per row: a row slice is 1 KB");
  static_assert(T <= 16 && S * T <= 256, "wave masks fit 16 bits, super-tile masks 8 words");
  static_assert(P <= 32 && P % S == 0 && (P & (P - 1)) == 0, "a stage's masks and ids fit one per lane");
  static_assert(NSLOT * P <= 192, "ids read ahead stay inside the plan's padding");
  constexpr bool DOC = DISP != kStRowMajor;   // masks from the plan's per-stage document words
  constexpr bool ROT = DISP == kStDocRotated;
  static_assert(!ROT || NSLOT == 2, "the rotated sweep tracks the next two stages");
  constexpr int64_t WN = 64 * K;      // neurons per slice
  constexpr int D = S * T;            // documents per super-tile
  constexpr int MW = (D + 31) / 32;   // mask words per union entry
  constexpr int RPW = P / S;          // rows each wave loads per stage
  constexpr int OPS = RPW + 1;        // loads per wave per stage (rows + mask words)
  __shared__ u32x4 ring[NSLOT][P][64];      // row slices
  __shared__ uint32_t mring[NSLOT][S][64];  // per wave: its mask word of each entry

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // XCD-contiguous super-tile ranges (see k_search)
  int64_t st, c;
  if (a.round_wgs) {
    // one round of one slice: every workgroup of the launch is resident at
    // once, so the round's super-tiles start together and sweep their
    // ascending unions side by side (each XCD's L2 holds the rows of the
    // feature range they share); XCD x takes the next round_wgs super-tiles
    // of its own contiguous range
    const int64_t j = blockIdx.x / kXcds;
    if (a.round_base + j >= a.xcd_span) return;
    st = (blockIdx.x % kXcds) * a.xcd_span + a.round_base + j;
    c = a.slice_base;
  } else if (a.chunk_slices > 1) {
    uint64_t u, sl;
    chunked_block(static_cast<uint64_t>(blockIdx.y) * gridDim.x + blockIdx.x, gridDim.x, gridDim.y,
                  static_cast<uint64_t>(a.chunk_slices), &u, &sl);
    st = static_cast<int64_t>(u);
    c = static_cast<int64_t>(sl);
  } else {
    const uint32_t per_xcd = gridDim.x / kXcds;
    st = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
    c = blockIdx.y;
  }
  if (st >= a.ntiles) return;  // whole workgroup: no barrier is skipped by part of it

  const int64_t n0 = c * WN;
  float acc[T][K];
#pragma unroll
  for (int s = 0; s < T; ++s)
#pragma unroll
    for (int k = 0; k < K; ++k) acc[s][k] = 0.f;

  // lanes past the last neuron re-read the last 128-bit group holding one, so
  // no load leaves [0, round_up(N, E)) of its row
  const int64_t o = E * lane;
  const int64_t nv = (a.N + E - 1) / E * E;
  const uint32_t offb = static_cast<uint32_t>(sizeof(WT) * (n0 + o < nv ? o : nv - E - n0));
  const char* __restrict__ Wn = reinterpret_cast<const char*>(static_cast<const WT*>(a.W) + n0) + offb;
  const int64_t ldw_b = a.ldw * static_cast<int64_t>(sizeof(WT));
  const int32_t u0 = a.tile_offset[st];
  const int32_t cnt = a.tile_count[st];
  // The plan pads its feature and mask arrays by 256 entries, so every read
  // of a whole stage (or of the ids NSLOT-1 stages ahead) stays inside it.
  // (The prologue reads ids through the constant address space: scalar loads,
  // which the vector-memory waits of the ring never drain.)
  typedef const __attribute__((address_space(4))) int32_t* const_i32;
  const const_i32 feat = (const_i32)(a.union_feat + u0);
  const int mword = (wave * T) >> 5;
  const int mshift = (wave * T) & 31;
  constexpr uint32_t kWaveBits = (1u << T) - 1u;
  // Each stage's dword load carries, per lane: lanes r < P the wave's mask
  // word of entry r of the stage; lanes P + r the feature id of entry r of the
  // stage NSLOT-1 later (so the row loads issued after a stage's barrier need
  // no scalar load); other lanes repeat lane r & (P-1)'s word.  With the
  // document-major dispatch (masks from the plan's stage words) only the id
  // lanes of the wave's own rows load: fewer addresses for the texture
  // addresser per stage (1.5% faster at 512^2; scalar loads of those ids a
  // stage ahead, in place of the dword load, were 3% slower).
  const bool id_lane = lane >= P && lane < 2 * P;
  const bool id_mine = lane >= P + wave * RPW && lane < P + wave * RPW + RPW;
  const uint32_t* __restrict__ dsrc =
      id_lane ? reinterpret_cast<const uint32_t*>(a.union_feat + u0 + (NSLOT - 1) * P + (lane - P))
              : a.union_mask + (static_cast<int64_t>(u0) + (lane & (P - 1))) * MW + mword;
  const int64_t dstride = id_lane ? P : static_cast<int64_t>(P) * MW;  // words per stage
  // rotated sweep: id lanes load entry lane - P of a stage from here
  const uint32_t* __restrict__ idl = reinterpret_cast<const uint32_t*>(a.union_feat + u0 + (id_lane ? lane - P : 0));
  const int32_t nstages = (cnt + P - 1) / P;
  // Rotated sweep: the phase of this super-tile.  An XCD starts its
  // super-tiles in tile order (one neuron slice after another) with about
  // a.phase_wgs of them running at once; taking the plan's nonzeros as the
  // measure of a super-tile's work, one starts when the XCD has done the work
  // of those before it less the work in flight, so its start time in units
  // of one super-tile's lifetime is, mod 1, the work of the range's earlier
  // super-tiles over phase_wgs times the range's mean work per super-tile.
  // The sweep starts that fraction of the way into the union.  The phase
  // depends on the plan and the launch's tile grid only (not on the slice),
  // so column ranges of one codebook still see the same order.
  int32_t s0 = 0;
  if (ROT && nstages > 1) {
    const int64_t per_xcd = gridDim.x / kXcds;
    const int64_t first = (blockIdx.x % kXcds) * per_xcd;
    const int64_t end = first + per_xcd < a.ntiles ? first + per_xcd : a.ntiles;
    const uint64_t o_first = static_cast<uint32_t>(a.tile_offset[first]);
    const uint64_t work = static_cast<uint32_t>(a.tile_offset[end]) - o_first;  // >= cnt > 0
    const uint64_t nx = static_cast<uint64_t>(end - first);
    const uint64_t den = static_cast<uint64_t>(a.phase_wgs) * work;             // < 2^41
    const uint64_t num = (static_cast<uint32_t>(u0) - o_first) * nx % den;      // product < 2^52
    const uint64_t ph = (num << 20) / den;                                      // phase in 2^-20
    s0 = __builtin_amdgcn_readfirstlane(static_cast<int32_t>((ph * static_cast<uint64_t>(nstages)) >> 20));
  }
  // stages of sequence steps 1 and 2 (rotated sweep; advanced one per step)
  int32_t a1 = s0 + 1 >= nstages ? s0 + 1 - nstages : s0 + 1;
  int32_t a2 = a1 + 1 >= nstages ? a1 + 1 - nstages : a1 + 1;
  // document-major stage masks (P = 16 entries per stage): stage q's word of
  // document j is 16-bit word j at mask word (u0 + q * P) * MW; this wave's
  // T words are T / 2 consecutive 32-bit words
  typedef const __attribute__((address_space(4))) uint32_t* const_u32;
  const const_u32 smask = (const_u32)(a.union_mask + static_cast<int64_t>(u0) * MW) + wave * (T / 2);
  constexpr int SW = T / 2;   // 32-bit words of stage masks per wave and stage
  uint32_t dmw[SW];
  if (DOC) {
    static_assert(P == 16, "document-major stage masks hold 16 entries");
#pragma unroll
    for (int k = 0; k < SW; ++k) dmw[k] = nstages > 0 ? smask[(ROT ? s0 * P * MW : 0) + k] : 0u;
  }
  const uint32_t ring0 = lds_offset(&ring[0][0][0]) + static_cast<uint32_t>(wave * RPW * 1024);
  const uint32_t mring0 = lds_offset(&mring[0][0][0]) + static_cast<uint32_t>(wave * 256);

  if (nstages > 0) {
    // stage q into slot q % NSLOT: this wave's rows (feature ids fid[i]), then
    // its dword load (mask words, ids of stage q + NSLOT - 1)
#define SOM_ST_ISSUE(q, fid)                                                                  \
  {                                                                                           \
    const int32_t q_ = (q);                                                                   \
    const uint32_t slot_ = static_cast<uint32_t>(q_ % NSLOT);                                 \
    _Pragma("unroll") for (int i = 0; i < RPW; ++i) {                                         \
      const int32_t e = (ROT ? s0 : q_) * P + wave * RPW + i; /* ROT: prologue step 0 only */ \
      const int64_t f = e < cnt ? (fid)[i] : 0;                                               \
      dma_b128(Wn + f * ldw_b, ring0 + slot_ * (P * 1024) + static_cast<uint32_t>(i * 1024)); \
    }                                                                                         \
    if (!DOC || id_mine) dma_b32(ROT ? idl + a1 * P : dsrc + q_ * dstride, mring0 + slot_ * (S * 256)); \
  }
#pragma unroll
    for (int q = 0; q < NSLOT - 1; ++q) {
      if (q < nstages) {
        int32_t fid[RPW];
#pragma unroll
        for (int i = 0; i < RPW; ++i) fid[i] = feat[(ROT ? s0 : q) * P + wave * RPW + i];
        SOM_ST_ISSUE(q, fid)
      }
    }
    if constexpr (DOC) {
      static_assert(NSLOT == 2, "document-major: a two-slot ring");
      // LDS byte offsets of the slot being added (the other slot receives the
      // next stage): 0 or one slot, swapped after every stage
      constexpr uint32_t kRingSlot = P * 1024, kMaskSlot = S * 256;
      uint32_t rcur = 0, mcur = 0;
      const uint32_t ring_lane = lds_offset(&ring[0][0][lane]);
      const uint32_t mring_lane = lds_offset(&mring[0][wave][lane]);
      // this wave's adds of the stage in the slot at ring offset rb
      auto add_stage = [&](uint32_t rb) {
        uint32_t cur[SW];
#pragma unroll
        for (int k = 0; k < SW; ++k) cur[k] = dmw[k];
        if constexpr (sizeof(WT) == 4 && K == 4 && T == 8) {
          const uint32_t vbase = ring_lane + rb;
          add_stage_8docs_f32(acc, cur, vbase);
        } else {
          const int slot = rb ? 1 : 0;
#pragma unroll
          for (int sd = 0; sd < T; ++sd) {
            // the entries of the stage that document sd of this wave holds
            uint32_t dm = (cur[sd >> 1] >> ((sd & 1) * 16)) & 0xffffu;
            while (dm) {
              const int r = __builtin_ctz(dm);
              dm &= dm - 1;
              float4 wf[K / 4];
              widen_v<WT>(ring[slot][r][lane], wf);
#pragma unroll
              for (int qq = 0; qq < K / 4; ++qq) {
                acc[sd][4 * qq + 0] += wf[qq].x;
                acc[sd][4 * qq + 1] += wf[qq].y;
                acc[sd][4 * qq + 2] += wf[qq].z;
                acc[sd][4 * qq + 3] += wf[qq].w;
              }
            }
          }
        }
      };
      // every stage but the last issues the next one; the last is peeled off
      for (int32_t s = 0; s + 1 < nstages; ++s) {
        vm_wait<0>();   // this wave's loads of stage s have landed
        lds_barrier();  // stage s visible to all waves; every wave is done with stage s-1
        const uint32_t w = *reinterpret_cast<const __attribute__((address_space(3))) uint32_t*>(
            static_cast<uintptr_t>(mring_lane + mcur));
        // the next stage: its rows' byte offsets computed once on the id
        // lanes (lane P + r holds entry r's feature id; past the union: row
        // 0), then moved to scalar registers one row at a time
        const int32_t qa = ROT ? a1 : s + 1;
        const bool live = id_lane && qa * P + (lane - P) < cnt;
        const uint64_t off = static_cast<uint64_t>(w & (live ? ~0u : 0u)) * static_cast<uint64_t>(ldw_b);
#pragma unroll
        for (int i = 0; i < RPW; ++i) {
          const int src = P + wave * RPW + i;
          const uint64_t o = (static_cast<uint64_t>(static_cast<uint32_t>(
                                 __builtin_amdgcn_readlane(static_cast<int>(off >> 32), src))) << 32) |
                             static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(off), src));
          dma_b128(Wn + o, ring0 + (kRingSlot - rcur) + static_cast<uint32_t>(i * 1024));
        }
        if (id_mine) dma_b32(ROT ? idl + a2 * P : dsrc + (s + 1) * dstride, mring0 + (kMaskSlot - mcur));
        add_stage(rcur);
        // the next stage's words, loaded now (their wait falls on the next
        // stage's first LDS read, after its barrier)
#pragma unroll
        for (int k = 0; k < SW; ++k)
          dmw[k] = reinterpret_cast<const_u32>(reinterpret_cast<const __attribute__((address_space(4))) char*>(smask) +
                                              static_cast<uint32_t>(qa) * (P * MW * 4))[k];
        if (ROT) {
          const int32_t n2 = a2 + 1;
          a1 = a2;
          a2 = n2 == nstages ? 0 : n2;
        }
        rcur = kRingSlot - rcur;
        mcur = kMaskSlot - mcur;
      }
      vm_wait<0>();
      lds_barrier();
      add_stage(rcur);
    } else {
    for (int32_t s = 0; s < nstages; ++s) {
      // this wave's stages issued after s: min(nstages - 1, s + NSLOT - 2) - s
      const int32_t later = (nstages - 1 < s + NSLOT - 2 ? nstages - 1 : s + NSLOT - 2) - s;
      wait_stages<OPS, NSLOT>(later);
      lds_barrier();  // stage s visible to all waves; every wave is done with stage s-1
      const int slot = s % NSLOT;
      const uint32_t w = mring[slot][wave][lane];
      if (s + NSLOT - 1 < nstages) {
        const int32_t q = s + NSLOT - 1;
        int32_t fid[RPW];
#pragma unroll
        for (int i = 0; i < RPW; ++i) fid[i] = __builtin_amdgcn_readlane(static_cast<int>(w), P + wave * RPW + i);
        SOM_ST_ISSUE(q, fid)
      }
      const uint32_t m_cur = (lane < P && s * P + lane < cnt) ? (w >> mshift) & kWaveBits : 0u;
      // this wave's needed entries of stage s, visited in ascending order
      uint64_t need = __ballot(m_cur != 0u);
      if (need) {
        int r = __builtin_ctzll(need);
        need &= need - 1;
        u32x4 cur = ring[slot][r][lane];
        uint32_t mc = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(m_cur), r));
        while (need) {
          const int r2 = __builtin_ctzll(need);
          need &= need - 1;
          const u32x4 nxt = ring[slot][r2][lane];
          const uint32_t mn = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(m_cur), r2));
          float4 wf[K / 4];
          widen_v<WT>(cur, wf);
          add_row<T, K, kMaskBranch>(acc, wf, mc);
          cur = nxt;
          mc = mn;
        }
        float4 wf[K / 4];
        widen_v<WT>(cur, wf);
        add_row<T, K, kMaskBranch>(acc, wf, mc);
      }
    }
    }
#undef SOM_ST_ISSUE
  }

  epilogue<WT, T, K>(a, acc, st * D + wave * T, n0, lane);
}

template <typename WT, int T, int K, int S>
hipError_t launch_st(const SearchArgs& a, hipStream_t stream) {
  // mask_mode: 1 = row-major dispatch, 2 = document-major
  // 16-entry stages in a ring of two: 32 KB of rows per workgroup, so four
  // workgroups of eight 8-document waves share a CU.  Measured on the 512^2
  // map (fp32, 262,144 documents): the number of waves a CU can interleave
  // decides the speed (each stage ends in a barrier that waits for the wave
  // with the most rows, and a wave's adds form a serial chain); 32-entry
  // stages, deeper rings and 16-document waves were slower.
  constexpr int P = 16;
  constexpr int NSLOT = 2;
  if (a.schedule == 2) {
    // round-synchronised launches: per slice, rounds of R super-tiles per
    // XCD, R = the workgroups one XCD holds at once (its CUs times the
    // kernel's occupancy per CU), so a launch's workgroups all start together
    const void* fn = a.mask_mode == 2 ? reinterpret_cast<const void*>(k_search_st<WT, T, K, S, P, NSLOT, kStDocMajor>)
                                      : reinterpret_cast<const void*>(k_search_st<WT, T, K, S, P, NSLOT, kStRowMajor>);
    int per_cu = 0, dev = 0, cus = 0;
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, S * 64, 0);
    if (e != hipSuccess) return e;
    e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    const int R = per_cu * cus / static_cast<int>(kXcds) > 0 ? per_cu * cus / static_cast<int>(kXcds) : 1;
    SearchArgs b = a;
    b.round_wgs = R;
    b.xcd_span = (a.ntiles + kXcds - 1) / kXcds;
    const int64_t rounds = (b.xcd_span + R - 1) / R;
    const dim3 grid(static_cast<uint32_t>(kXcds * R), 1);
    for (int64_t c = 0; c < a.nchunks; ++c) {
      b.slice_base = c;
      for (int64_t r = 0; r < rounds; ++r) {
        b.round_base = r * R;
        if (a.mask_mode == 2)
          hipLaunchKernelGGL((k_search_st<WT, T, K, S, P, NSLOT, kStDocMajor>), grid, dim3(S * 64), 0, stream, b);
        else
          hipLaunchKernelGGL((k_search_st<WT, T, K, S, P, NSLOT, kStRowMajor>), grid, dim3(S * 64), 0, stream, b);
      }
    }
    return hipGetLastError();
  }
  const dim3 grid(static_cast<uint32_t>((a.ntiles + kXcds - 1) / kXcds * kXcds), static_cast<uint32_t>(a.nchunks));
  if (a.mask_mode == 2 && a.rotate) {
    SearchArgs b = a;
    const hipError_t e = st_phase_wgs(T, S, &b.phase_wgs);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((k_search_st<WT, T, K, S, P, NSLOT, kStDocRotated>), grid, dim3(S * 64), 0, stream, b);
    return hipGetLastError();
  }
  if (a.mask_mode == 2)
    hipLaunchKernelGGL((k_search_st<WT, T, K, S, P, NSLOT, kStDocMajor>), grid, dim3(S * 64), 0, stream, a);
  else
    hipLaunchKernelGGL((k_search_st<WT, T, K, S, P, NSLOT, kStRowMajor>), grid, dim3(S * 64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace
}  // namespace som
