// Steps 3 and 4 for bf16 and fp8-e4m3 corpora: score every distinct query
// against the corpus on the matrix cores and keep the k best rows per query
// and corpus slice.
//
// HeraSys runs one retrieval per fused node (Sec. 3.3 (I)) and batches ready
// nodes of the same type (Appendix A, batching constraint); a retrieval
// node's result is its Top-K chunks (Eq. 2 parameters; Sec. 4.1 workloads).
// Here the batch is the n_u distinct queries and the retrieval is an exact
// inner product, s[u, c] = scale_c * sum_j Q[u, j] C[c, j], accumulated in
// fp32.
//
// Work decomposition: a persistent grid, one workgroup of four waves per CU.
// A work item is (query tile of 128, corpus slice); a slice is a run of
// tiles of 384 corpus rows.  Wave w owns rows [96w, 96w + 96) of a tile
// against all 128 queries: 3 x 4 blocks of v_mfma_f32_32x32x16_bf16 with the
// 192 fp32 accumulators in AGPRs (the rest of the register file holds two
// sets of operand fragments and the epilogue's working set without spills).
// Items of one slice get consecutive logical ids on one XCD, so the query
// tiles that read the same corpus rows share that XCD's L2.
//
// Operand staging: both operands stream through a ring of LDS stages (two
// for bf16, three for fp8), one K range of 64 per stage, written by
// buffer_load ... lds (asynchronous copies from global memory straight into
// LDS, no registers).  A bf16 corpus row contributes one 128-byte line per
// stage (fp8: 64 bytes).  Rows are stored in LDS as 16-byte pieces with an
// XOR swizzle so that fragment reads (ds_read_b128) are bank-conflict free.
// The query rows, and the corpus when it is given in the tiled layout, are
// kept in global memory in exactly that LDS order (tile_queries_kernel,
// tile_corpus_kernel), zero-padded past n_u, N and d, so every copy reads
// 1 KiB of consecutive bytes; a row-major corpus is copied as row pieces
// through a descriptor whose range covers the tile's valid rows (rows past N
// read as zeros).  Either way there are no bounds branches and no access
// outside the operands.  Inside one MFMA the K order is free as long as
// both operands agree; each lane takes the K slice that makes its fp8 corpus
// piece one 16-byte read.
//
// Synchronisation per stage: a wave copies, and alone reads, its own 96
// corpus rows of a stage, so it refills them as soon as its own reads of
// the stage's slot are complete (after the first of the four MFMA steps),
// without a barrier.  The query rows are shared by the four waves: after the
// third step the waves wait for their own copies of the next stage
// (s_waitcnt vmcnt with the number of younger copies), then one barrier,
// then the query rows of the stage ns ahead and the next stage's first
// fragments, overlapped with the last step.  The fences of __syncthreads are
// not used because they would wait for every copy in flight.
//
// Top-k (fused, scores never reach memory), per tile: rows past N are
// masked and each lane screens its 16-score row blocks by their maximum
// (fp8: accumulator x row scale) against the query's threshold; only the
// blocks that reach it are examined, and their scores at or above it are
// appended to a small per-query LDS queue (one atomic per lane and block
// reserves the slots), merged into the query's sorted k-list when a queue
// is due.  Thresholds come from lower bounds of the query's final k-th best
// score: the slice's own k-list; a seed, the k-th largest of the lane maxima
// of a first pass over the first tiles of the slices (at most 128 of them:
// a sample spread over the corpus); the order statistics of the slices
// finished so far; and the
// largest bound any slice of the query has published so far (a per-query
// array in the workspace, read asynchronously with each tile's copies).
// Keys order by (score desc, row asc): ties go to the lower
// corpus row independently of tile, slice or lane.
#include <mutex>
#include <type_traits>

#include "common.h"

namespace hs {

typedef __bf16 bf16x8m __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2m __attribute__((ext_vector_type(2)));
typedef float f32x16m __attribute__((ext_vector_type(16)));

constexpr int kMW = 4;                   // waves per workgroup (one per SIMD)
constexpr int kMT = kMW * 64;            // threads
constexpr int kMRB = 3;                  // 32-row blocks per wave
constexpr int kMQB = 4;                  // 32-query blocks per tile
constexpr int kMNC = kMW * 32 * kMRB;    // 384 corpus rows per tile
constexpr int kMMQ = 32 * kMQB;          // 128 queries per tile
constexpr int kMKC = 64;                 // K per ring stage (four 16-deep MFMA steps)
constexpr int kMQcap = 8;                // queue slots per query and round
constexpr int kMVals = 16 * kMRB;        // scores per lane and query per tile
constexpr int kMLanesQ = kMW * 2;        // lanes holding one query in a tile

// Seed pass sample: the lane maxima of the first T tiles of every slice (at
// most kSeedMax of them per query).  T is one for k <= 48.  For larger k the
// k-th largest lane maximum of one tile per slice is a weak bound (k is then a
// sizeable fraction of the sample): a sample of M rows lets about N k / M rows
// of the corpus pass it, each a list insertion, and with many slices the
// lists do not fill before their slice ends, so their own minima never take
// over.  T therefore grows to 20 as long as the sample stays within 1/16 of
// the slice's tiles and within kSeedMax values.
constexpr int kSeedMax = 16384;
constexpr int kSeedTilesMax = 20;
__host__ __device__ __forceinline__ int seed_tiles(int k, int64_t ntiles, int64_t S) {
  if (k <= 48 || S < 1) return 1;
  int64_t t = ntiles / (S * 16);
  const int64_t room = kSeedMax / (S * kMLanesQ);
  if (t > room) t = room;
  if (t > kSeedTilesMax) t = kSeedTilesMax;
  return t < 1 ? 1 : (int)t;
}
// Slices that take part in the seed sample: one in every seed_stride(S), at
// most kSeedSlices of them.  A single query tile runs as up to 256 slices, and
// the seed pass (one tile per workgroup, all at once) then reads that many
// tiles of the corpus; half of them are as good a sample for the seed.
constexpr int kSeedSlices = 128;
__host__ __device__ __forceinline__ int64_t seed_stride(int64_t S) {
  return S > kSeedSlices ? (S + kSeedSlices - 1) / kSeedSlices : 1;
}
constexpr int kMSplitMaxSK = 8192;       // bound on S*k (merge list length)
constexpr int kMRowsW = 32 * kMRB;       // rows per wave in a tile
constexpr int kMSS = kMNC + 128 - kMRowsW;  // row-scale slot stride (floats): the
                                         // last wave's two 64-row copies overhang
constexpr int kMLdsMax = 160 * 1024;     // LDS per workgroup on gfx950
constexpr int kMGridMax = 512;           // persistent grid never exceeds this
constexpr int kMGts = kMMQ + 32;         // shared-threshold slot stride (entries): the
                                         // last wave's 64-entry copy overhangs

template <bool FP8>
struct Geo {
  static constexpr int esz = FP8 ? 1 : 2;
  static constexpr int arow = kMKC * esz;         // bytes of one corpus row per stage
  static constexpr int abytes = kMNC * arow;
  static constexpr int brow = kMKC * 2;           // bytes of one query row per stage
  static constexpr int bbytes = kMMQ * brow;
  static constexpr int stage = abytes + bbytes;
  static constexpr int ns = FP8 ? 3 : 2;          // ring stages
  static constexpr int nsc = FP8 ? ns + 1 : 0;    // row-scale slots (tiles in flight)
  static constexpr int ngt = ns + 1;              // shared-threshold slots (tiles in flight)
  static constexpr int adma = abytes / 1024 / kMW;  // 1 KiB copies per wave and stage
  static constexpr int bdma = bbytes / 1024 / kMW;
  static constexpr int ldma = adma + bdma;        // copies per wave and stage (scales aside)
  static constexpr int apieces = arow / 16;       // 16-byte pieces of a corpus row stage
  static constexpr int bpieces = brow / 16;
};

// Slot of 16-byte piece p in a row of P pieces.  gfx950's LDS serves a
// ds_read_b128 16 lanes at a time over 64 banks (256 bytes); the fragment
// reads have 16 consecutive rows read the same piece, so the 16 / P rows that
// share a 256-byte window must get distinct slots, for every p: the slot is p
// XOR the row's window number (mod P).  Only row mod 16 matters.
template <int P>
__device__ __forceinline__ int swz_slot(int p, int row) {
  return p ^ ((row / (16 / P)) & (P - 1));
}

constexpr int kMTail = 16;   // list entries kept in LDS when the lists are global

// Order statistics a finished item publishes per query: level l holds the
// ordered score of the ceil(k / r)-th best key of the slice's final list,
// r = 2^l, l < kLvl (0 where the list is shorter).  If r slices publish level-l
// values of at least x, those slices hold r * ceil(k / r) >= k distinct
// rows scoring at least x, so the r-th largest level-l value over the
// slices is a lower bound of the query's k-th best score.  An item starts
// by raising the query's shared threshold to the best such bound over the
// slices finished so far.
constexpr int kLvl = 5;
constexpr int kMWarmBytes = kMW * kMMQ * 4;   // per-wave warm-up minima (alias the queue)
static_assert(kMWarmBytes <= kMMQ * kMQcap * 8, "warm-up minima fit in the queue");

__host__ __device__ constexpr int mfma_lds_bytes(bool fp8, bool lds_lists, int k) {
  return (fp8 ? Geo<true>::ns * Geo<true>::stage + Geo<true>::nsc * kMSS * 4 +
                    Geo<true>::ngt * kMGts * 4
              : Geo<false>::ns * Geo<false>::stage + Geo<false>::ngt * kMGts * 4) +
         kMMQ * kMQcap * 8 + kMMQ * (4 + 4 + 4 + 8 + 4) + 16 +
         (lds_lists ? kMMQ * k * 8 : kMMQ * kMTail * 8);
}
// k-lists of up to kMTail entries always fit in LDS, so global lists (which
// keep kMTail entries in LDS) always have k > kMTail; and the global-list
// layout fits for every k.
static_assert(mfma_lds_bytes(false, true, kMTail) <= 160 * 1024 &&
                  mfma_lds_bytes(true, true, kMTail) <= 160 * 1024,
              "short k-lists fit in LDS");
static_assert(mfma_lds_bytes(false, false, 0) <= 160 * 1024 &&
                  mfma_lds_bytes(true, false, 0) <= 160 * 1024,
              "global-list layout fits in LDS");

// Warm-up groups per lane and query: the kMVals scores a lane holds for one
// query are cut into gpl groups so that kMLanesQ * gpl >= k group maxima
// exist.  0 = no warm-up (k too large for one tile).
__host__ __device__ constexpr int mwarm_groups(int k) {
  int g = 1;
  while (g <= kMVals && kMLanesQ * g < k) g <<= 1;
  return g <= kMVals ? g : 0;
}

__device__ __forceinline__ void cvt8_fp8_bf16(uint32_t lo, uint32_t hi, bf16x8m &out) {
  // exact e4m3 -> bf16 (every e4m3 value is representable in bf16)
  bf16x2m a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(lo, 1.0f, false);
  bf16x2m b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(lo, 1.0f, true);
  bf16x2m c = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(hi, 1.0f, false);
  bf16x2m e = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(hi, 1.0f, true);
  uint4 v = make_uint4(__builtin_bit_cast(uint32_t, a), __builtin_bit_cast(uint32_t, b),
                       __builtin_bit_cast(uint32_t, c), __builtin_bit_cast(uint32_t, e));
  out = __builtin_bit_cast(bf16x8m, v);
}

// Barrier for LDS data: this wave's LDS operations complete, then s_barrier.
// No memory fence, so copies into the ring stay in flight across it.
__device__ __forceinline__ void bar_lds() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// Wait until at most n of this wave's vector-memory operations are pending
// (they complete in issue order).  n is one of the few values a ring depth
// can produce.
__device__ __forceinline__ void wait_vm(int n) {
  __builtin_amdgcn_sched_barrier(0);
  switch (n) {
#define HS_VM_CASE(x) \
  case x: asm volatile("s_waitcnt vmcnt(" #x ")" ::: "memory"); break;
    HS_VM_CASE(1) HS_VM_CASE(2) HS_VM_CASE(3) HS_VM_CASE(4) HS_VM_CASE(5) HS_VM_CASE(6)
    HS_VM_CASE(7) HS_VM_CASE(8) HS_VM_CASE(9) HS_VM_CASE(10) HS_VM_CASE(11) HS_VM_CASE(12)
    HS_VM_CASE(13) HS_VM_CASE(14) HS_VM_CASE(15) HS_VM_CASE(16) HS_VM_CASE(17) HS_VM_CASE(18)
    HS_VM_CASE(19) HS_VM_CASE(20) HS_VM_CASE(21) HS_VM_CASE(22) HS_VM_CASE(23) HS_VM_CASE(24)
    HS_VM_CASE(25) HS_VM_CASE(26) HS_VM_CASE(27) HS_VM_CASE(28) HS_VM_CASE(29) HS_VM_CASE(30)
    HS_VM_CASE(31) HS_VM_CASE(32)
#undef HS_VM_CASE
    default: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
  }
  __builtin_amdgcn_sched_barrier(0);
}

// Buffer descriptor (raw, stride 0) over [base, base + bytes): loads at
// offsets past `bytes` return zeros and touch no memory.
typedef int i32x4m __attribute__((ext_vector_type(4)));
__device__ __forceinline__ i32x4m make_rsrc(const void *base, uint32_t bytes) {
  // (the operands are wave-uniform; readfirstlane puts them in SGPRs)
  const uint64_t p = (uint64_t)base;
  i32x4m r;
  r.x = __builtin_amdgcn_readfirstlane((int)(uint32_t)p);
  r.y = __builtin_amdgcn_readfirstlane((int)((uint32_t)(p >> 32) & 0xFFFFu));
  r.z = __builtin_amdgcn_readfirstlane((int)bytes);
  r.w = 0x00020000;
  return r;
}

// Asynchronous copies global -> LDS (buffer_load ... lds): lane l writes its
// 16 (or 4) bytes at lds + 16 l (or 4 l).  They are issued from inline asm
// on purpose: the compiler cannot tell which LDS bytes such a copy writes,
// so for the builtin form it drains every copy in flight before any later
// LDS read, which would defeat the ring.  The kernel orders the copies
// itself (wait_vm, then a barrier).  M0 holds the LDS base; the compiler
// reserves M0 and sets it before each of its own uses, so overwriting it
// here is harmless.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(i32x4m rsrc, const void *lds, uint32_t voff) {
  const uint32_t l = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :: "s"(l), "v"(voff), "s"(rsrc) : "memory", "m0");
}
__device__ __forceinline__ void dma4(i32x4m rsrc, const void *lds, uint32_t voff) {
  const uint32_t l = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, 0 offen lds"
               :: "s"(l), "v"(voff), "s"(rsrc) : "memory", "m0");
}
__device__ __forceinline__ void dma16s(i32x4m rsrc, uint32_t lds, uint32_t voff) {
  const uint32_t l = __builtin_amdgcn_readfirstlane(lds);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :: "s"(l), "v"(voff), "s"(rsrc) : "memory", "m0");
}
#pragma clang diagnostic pop

struct MfmaArgs {
  const void *q;
  const void *corpus;
  const float *scale;
  int64_t N, d;
  int k;
  int64_t n_unique;
  const int64_t *n_unique_dev;
  int64_t cap;
  int grid;
  int tiled;        // corpus in the tiled layout (tile_corpus_kernel), else row-major
  uint64_t *part;
  uint32_t *gthr;   // [cap] per-query shared thresholds (ordered score, 0 = none)
  uint32_t *lmax;   // [n_u][S][T][8] lane maxima of the seed pass (ordered scores)
  uint32_t *lvl;    // [n_u][kLvl][S] order statistics of finished items (ordered scores)
};

// Fragments of one half stage (two 16-deep steps).  The K order inside a
// stage is permuted identically for both operands: step t in 0..3 and lane
// half h take elements [32h + 8t, 32h + 8t + 8), so that one 16-byte fp8
// corpus piece feeds two consecutive steps.
template <bool FP8, int NQB>
struct Frag {
  // bf16: A pieces [step][rb]; fp8: raw 16-byte pieces [rb] (both steps)
  uint4 a[FP8 ? 1 : 2][kMRB];
  uint4 b[2][NQB];
  // ds_read_b128 operations that fill one Frag
  static constexpr int na = (FP8 ? 1 : 2) * kMRB;
  static constexpr int nreads = na + 2 * NQB;
};

// Read k (0 <= k < nreads) of half u of the stage in ring slot `st`: the A
// pieces first (step-major), then the B pieces (step-major).
template <bool FP8, int NQB>
__device__ __forceinline__ void read_frag_piece(Frag<FP8, NQB> &f, const unsigned char *st,
                                                int wv, int c, int h, int u, int k) {
  using G = Geo<FP8>;
  using F = Frag<FP8, NQB>;
  if (k < F::na) {
    const int s = FP8 ? 0 : k / kMRB, rb = k % kMRB;
    const int slot = FP8 ? swz_slot<G::apieces>(2 * h + u, c)
                         : swz_slot<G::apieces>(4 * h + 2 * u + s, c);
    const unsigned char *abase = st + (wv * 32 * kMRB + c) * G::arow;
    f.a[s][rb] = *reinterpret_cast<const uint4 *>(abase + rb * 32 * G::arow + slot * 16);
  } else {
    const int s = (k - F::na) / NQB, qb = (k - F::na) % NQB;
    const int slot = swz_slot<G::bpieces>(4 * h + 2 * u + s, c);
    const unsigned char *bbase = st + G::abytes + c * G::brow;
    f.b[s][qb] = *reinterpret_cast<const uint4 *>(bbase + qb * 32 * G::brow + slot * 16);
  }
}

// Read half u of the stage in ring slot `st`.
template <bool FP8, int NQB>
__device__ __forceinline__ void read_frags(Frag<FP8, NQB> &f, const unsigned char *st, int wv,
                                           int c, int h, int u) {
#pragma unroll
  for (int k = 0; k < Frag<FP8, NQB>::nreads; ++k) read_frag_piece<FP8>(f, st, wv, c, h, u, k);
}

// Redefine the second step's operands of a half stage in place (no code):
// MFMAs that use them cannot then be moved above a preceding barrier.
typedef unsigned u32x4m __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void pin_u4(uint4 &v) {
  u32x4m t = __builtin_bit_cast(u32x4m, v);
  asm volatile("" : "+v"(t));
  v = __builtin_bit_cast(uint4, t);
}
template <bool FP8, int NQB>
__device__ __forceinline__ void pin_step1(Frag<FP8, NQB> &f) {
#pragma unroll
  for (int rb = 0; rb < kMRB; ++rb) pin_u4(f.a[FP8 ? 0 : 1][rb]);
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) pin_u4(f.b[1][qb]);
}

// One 16-deep MFMA step over the wave's kMRB x NQB blocks.
template <bool FP8, bool ZERO, int NQB>
__device__ __forceinline__ void mfma_step(f32x16m (&acc)[kMRB][NQB], const Frag<FP8, NQB> &f,
                                          int s) {
  bf16x8m av[kMRB];
#pragma unroll
  for (int rb = 0; rb < kMRB; ++rb) {
    if constexpr (FP8) {
      const uint4 v = f.a[0][rb];
      if (s == 0) cvt8_fp8_bf16(v.x, v.y, av[rb]);
      else cvt8_fp8_bf16(v.z, v.w, av[rb]);
    } else {
      av[rb] = __builtin_bit_cast(bf16x8m, f.a[s][rb]);
    }
  }
  const f32x16m zero = {};
#pragma unroll
  for (int rb = 0; rb < kMRB; ++rb)
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb)
      acc[rb][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
          av[rb], __builtin_bit_cast(bf16x8m, f.b[s][qb]), ZERO ? zero : acc[rb][qb], 0, 0, 0);
}

template <bool FP8, bool ZERO, int NOPS, int NQB, typename Op>
__device__ __forceinline__ void mfma_step_il(f32x16m (&acc)[kMRB][NQB], const Frag<FP8, NQB> &f,
                                             int s, Op &&op) {
  bf16x8m av[kMRB];
#pragma unroll
  for (int rb = 0; rb < kMRB; ++rb) {
    if constexpr (FP8) {
      const uint4 v = f.a[0][rb];
      if (s == 0) cvt8_fp8_bf16(v.x, v.y, av[rb]);
      else cvt8_fp8_bf16(v.z, v.w, av[rb]);
    } else {
      av[rb] = __builtin_bit_cast(bf16x8m, f.a[s][rb]);
    }
  }
  const f32x16m zero = {};
  constexpr int NM = kMRB * NQB;
#pragma unroll
  for (int i = 0; i < NM; ++i) {
    const int rb = i / NQB, qb = i % NQB;
    acc[rb][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
        av[rb], __builtin_bit_cast(bf16x8m, f.b[s][qb]), ZERO ? zero : acc[rb][qb], 0, 0, 0);
#pragma unroll
    for (int k = i * NOPS / NM; k < (i + 1) * NOPS / NM; ++k) op(k);
    __builtin_amdgcn_sched_barrier(0);
  }
}

struct MLds {
  unsigned char *ring;
  float *sscale;     // [nsc][kMSS] row scales of the tiles in flight (fp8)
  uint32_t *gtl;     // [ngt][kMGts] shared thresholds of the tiles in flight
  uint64_t *queue;   // [MQ][kMQcap] keys queued this round
  int32_t *qcount;   // [MQ] keys queued (may exceed kMQcap: overflow)
  float *thr0;       // [MQ] warm-up threshold of the item
  float *thr;        // [MQ] current threshold
  uint32_t *pub;     // [MQ] last threshold published to the shared array
  uint64_t *lmin;    // [MQ] last key of the sorted list when full, else its fill count
  float *warm;       // [kMW][MQ] per-wave minima of group maxima (aliases queue)
  int32_t *flags;    // [1] overflow epoch, [2] merge-due epoch
  uint64_t *lists;   // [MQ][k] or nullptr (lists in the global partial buffer)
  uint64_t *tail;    // [MQ][kMTail] last entries of the global lists, or nullptr
};

template <bool FP8, bool LDS_LISTS>
__device__ __forceinline__ MLds carve_mlds(unsigned char *p, int k) {
  using G = Geo<FP8>;
  MLds L;
  L.ring = p; p += G::ns * G::stage;
  L.sscale = reinterpret_cast<float *>(p); p += G::nsc * kMSS * 4;
  L.gtl = reinterpret_cast<uint32_t *>(p); p += G::ngt * kMGts * 4;
  L.queue = reinterpret_cast<uint64_t *>(p);
  L.warm = reinterpret_cast<float *>(p);   // (used before the queue in an epilogue)
  p += kMMQ * kMQcap * 8;
  L.lmin = reinterpret_cast<uint64_t *>(p); p += kMMQ * 8;
  L.qcount = reinterpret_cast<int32_t *>(p); p += kMMQ * 4;
  L.thr0 = reinterpret_cast<float *>(p); p += kMMQ * 4;
  L.thr = reinterpret_cast<float *>(p); p += kMMQ * 4;
  L.pub = reinterpret_cast<uint32_t *>(p); p += kMMQ * 4;
  L.flags = reinterpret_cast<int32_t *>(p); p += 16;
  L.lists = LDS_LISTS ? reinterpret_cast<uint64_t *>(p) : nullptr;
  L.tail = LDS_LISTS ? nullptr : reinterpret_cast<uint64_t *>(p);
  (void)k;
  return L;
}

struct MItem {
  int qbase, qvalid, s;
  int64_t S;
  int T;   // tiles per slice of the seed pass sample
};

// Publish query t's threshold (a lower bound of its k-th best score over its
// slice, hence over the whole corpus) to the per-query shared array: every
// slice of the query filters with the largest bound any slice has reached.
__device__ __forceinline__ void publish_thr(const MLds &L, const MfmaArgs &a, const MItem &it,
                                            int t, float th) {
  if (!(th > -__builtin_inff())) return;
  const uint32_t o = ord_score(th);
  if (o > L.pub[t]) {
    L.pub[t] = o;
    atomicMax(a.gthr + it.qbase + t, o);
  }
}

// Keep t (descending) the R largest of the values offered so far.
template <int R>
__device__ __forceinline__ void offer_top(uint32_t (&t)[R], uint32_t x) {
#pragma unroll
  for (int u = 0; u < R; ++u) {
    const uint32_t hi = t[u] > x ? t[u] : x;
    x = t[u] > x ? x : t[u];
    t[u] = hi;
  }
}

// Best lower bound of a query's k-th best score from the order statistics
// its finished slices published: the largest over levels l of the 2^l-th
// largest level-l value over the S slices (0 if none).  lv = the query's
// [kLvl][S] row; device-scope loads (other workgroups publish), issued 8
// slices x kLvl levels at a time.
__device__ __forceinline__ uint32_t level_bound(const uint32_t *lv, int S) {
  static_assert(kLvl == 5, "one top buffer per level");
  uint32_t t0[1] = {0u}, t1[2] = {0u, 0u}, t2[4] = {}, t3[8] = {}, t4[16] = {};
  for (int s0 = 0; s0 < S; s0 += 8) {
    uint32_t v[kLvl][8];
#pragma unroll
    for (int l = 0; l < kLvl; ++l)
#pragma unroll
      for (int u = 0; u < 8; ++u)
        v[l][u] = s0 + u < S ? __hip_atomic_load(lv + l * S + s0 + u, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT)
                             : 0u;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      offer_top(t0, v[0][u]);
      offer_top(t1, v[1][u]);
      offer_top(t2, v[2][u]);
      offer_top(t3, v[3][u]);
      offer_top(t4, v[4][u]);
    }
  }
  uint32_t b = t0[0];
  b = t1[1] > b ? t1[1] : b;
  b = t2[3] > b ? t2[3] : b;
  b = t3[7] > b ? t3[7] : b;
  b = t4[15] > b ? t4[15] : b;
  return b;
}

// Merge the queued keys of query t into its k-list (one thread per query).
// The list is kept sorted in descending key order (empty slots are key 0 at
// the end), so its minimum is always the last entry and an insertion only
// shifts the entries it passes: near the threshold, where nearly every
// entrant lands, that is one or two steps.  A list in the global partial
// buffer keeps its last kMTail entries in LDS while the item runs (its head,
// positions [0, k - kMTail), stays in global memory): an insertion touches
// global memory only when its key climbs above that window.
template <bool LDS_LISTS>
__device__ __forceinline__ void merge_queue(const MLds &L, const MfmaArgs &a, const MItem &it,
                                            int t) {
  const int cnt = L.qcount[t];
  if (cnt <= 0) return;
  const int n = cnt < kMQcap ? cnt : kMQcap;
  const int k = a.k;
  const int hb = LDS_LISTS ? k : k - kMTail;   // first position held in the LDS tail
  uint64_t *l = LDS_LISTS ? L.lists + t * k
                          : a.part + ((int64_t)(it.qbase + t) * it.S + it.s) * k;
  uint64_t *tail = LDS_LISTS ? nullptr : L.tail + t * kMTail;
  auto get = [&](int i) -> uint64_t { return (!LDS_LISTS && i >= hb) ? tail[i - hb] : l[i]; };
  auto set = [&](int i, uint64_t v) {
    if (!LDS_LISTS && i >= hb)
      tail[i - hb] = v;
    else
      l[i] = v;
  };
  // lmin holds the list's last key once the list is full, else its fill
  // count (below 2^32, hence below every key: a real key's ordered score is
  // nonzero), so that an entrant of a list that is not full starts at the
  // first empty slot instead of climbing over the empty ones
  uint64_t mn = L.lmin[t];
  int fill = (mn >> 32) ? k : (int)mn;
  for (int e = 0; e < n; ++e) {
    const uint64_t key = L.queue[t * kMQcap + e];
    if (key > mn) {
      int i = fill < k ? fill : k - 1;   // the key's slot if no entry above is smaller
      if constexpr (LDS_LISTS) {
        while (i > 0) {
          const uint64_t prev = get(i - 1);
          if (prev > key) break;
          set(i, prev);
          --i;
        }
      } else {
        // climb in windows of 8 entries read together (independent global
        // loads): the window's entries above the key stay, the others move
        // down by one
        while (i > 0) {
          const int lo = i > 8 ? i - 8 : 0;
          uint64_t b[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) b[u] = lo + u < i ? get(lo + u) : 0ull;   // (0: not above)
          int above = 0;
#pragma unroll
          for (int u = 0; u < 8; ++u) above += b[u] > key ? 1 : 0;
#pragma unroll
          for (int u = 7; u >= 0; --u)
            if (u >= above && lo + u < i) set(lo + u + 1, b[u]);
          if (above > 0 || lo == 0) {
            i = lo + above;
            break;
          }
          i = lo;
        }
      }
      set(i, key);
      if (fill < k) ++fill;
      mn = fill == k ? get(k - 1) : (uint64_t)fill;
    }
  }
  L.lmin[t] = mn;
  const float tl = (mn >> 32) ? unord_score((uint32_t)(mn >> 32)) : -__builtin_inff();
  const float t0v = L.thr0[t];
  L.thr[t] = tl > t0v ? tl : t0v;
  publish_thr(L, a, it, t, L.thr[t]);
  L.qcount[t] = 0;
}

// Keep the accumulators in AGPRs and make the compiler forget any VGPR copy
// of them: the epilogue then reads each element where it is used instead of
// holding all 256 in VGPRs across its loops.
template <int NQB>
__device__ __forceinline__ void pin_acc(f32x16m (&acc)[kMRB][NQB]) {
#pragma unroll
  for (int rb = 0; rb < kMRB; ++rb)
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) asm volatile("" : "+a"(acc[rb][qb]));
}

// An opaque copy of a lane value: values derived from it are recomputed
// where they are used instead of being hoisted (and spilled) by the compiler.
__device__ __forceinline__ int opaque(int x) {
  asm volatile("" : "+v"(x));
  return x;
}

// Turns the tile's accumulators into scores in place, once per tile: the fp8
// row scale applied, NaN for rows past N (NaN fails every >= test and fmaxf
// ignores it).  Accumulator element (rb, qb, i) of a lane is row
// rb * 32 + 8 * (i / 4) + i % 4 counted from the lane's first row; `lim0` =
// number of valid rows from there.  Everything after reads the accumulators
// directly.
template <bool FP8, int NQB>
__device__ __forceinline__ void finish_scores(f32x16m (&acc)[kMRB][NQB], const float *ssc_lane,
                                              int lim0) {
  if constexpr (FP8) {
#pragma unroll
    for (int rb = 0; rb < kMRB; ++rb)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        // (an opaque offset keeps the compiler from loading all 48 scales
        // ahead of the multiplies)
        const float4 s4 = *reinterpret_cast<const float4 *>(ssc_lane + opaque(rb * 32 + 8 * j));
#pragma unroll
        for (int qb = 0; qb < NQB; ++qb) {
          acc[rb][qb][4 * j + 0] *= s4.x;
          acc[rb][qb][4 * j + 1] *= s4.y;
          acc[rb][qb][4 * j + 2] *= s4.z;
          acc[rb][qb][4 * j + 3] *= s4.w;
          asm volatile("" : "+a"(acc[rb][qb]));
        }
      }
  }
  if (lim0 < 32 * kMRB) {   // some of this lane's rows are past N
    const float nan = __builtin_nanf("");
#pragma unroll
    for (int rb = 0; rb < kMRB; ++rb)
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (rb * 32 + 8 * (i >> 2) + (i & 3) >= lim0) acc[rb][qb][i] = nan;
    pin_acc(acc);
  }
}
// NaN for the scores of rows past N (only for a tile that reaches past N).
template <int NQB>
__device__ __forceinline__ void mask_tail(f32x16m (&acc)[kMRB][NQB], int lim0) {
  if (lim0 < 32 * kMRB) {   // some of this lane's rows are past N
    const float nan = __builtin_nanf("");
#pragma unroll
    for (int rb = 0; rb < kMRB; ++rb)
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (rb * 32 + 8 * (i >> 2) + (i & 3) >= lim0) acc[rb][qb][i] = nan;
    pin_acc(acc);
  }
}

// The 16 fp8 row scales of row block rb of this lane (rows rb * 32 + 8 * (i /
// 4) + i % 4 from the lane's first row), or ones when the accumulators are
// already scaled.
template <bool FP8>
__device__ __forceinline__ void row_scales(float (&s16)[16], const float *ssc_lane, int rb,
                                           bool ones) {
  if constexpr (FP8) {
    if (!ones) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float4 s4 = *reinterpret_cast<const float4 *>(ssc_lane + rb * 32 + 8 * j);
        s16[4 * j + 0] = s4.x;
        s16[4 * j + 1] = s4.y;
        s16[4 * j + 2] = s4.z;
        s16[4 * j + 3] = s4.w;
      }
      return;
    }
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) s16[i] = 1.0f;
}


// Warm-up: per query, the smallest of this lane's group maxima (groups of
// SPAN consecutive scores), combined over the two lane halves and stored per
// wave.
template <int SPAN, int NQB>
__device__ __forceinline__ void warm_minima(const MLds &L, f32x16m (&acc)[kMRB][NQB], int wv,
                                            int c, int h) {
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    float mn = __builtin_inff(), m = -__builtin_inff();
#pragma unroll
    for (int rb = 0; rb < kMRB; ++rb)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        m = fmaxf(m, acc[rb][qb][i]);
        if ((rb * 16 + i + 1) % SPAN == 0) {
          mn = fminf(mn, m);
          m = -__builtin_inff();
        }
      }
    mn = fminf(mn, __shfl_xor(mn, 32));
    if (h == 0) L.warm[wv * kMMQ + qb * 32 + c] = mn;
  }
}

// Seed pass: each lane's best score of the tile for each of its queries, as
// an ordered score, to lmax[((query * S + slice) * T + t) * 8 + lane-of-query]
// for the slice's t-th sampled tile (T tiles per slice).  These
// are scores of distinct corpus rows, so the k-th largest of all of a
// query's lane maxima (over all slices) is a lower bound of its k-th best
// score over the whole corpus.
template <bool FP8, int NQB>
__device__ __forceinline__ void mtile_lane_maxima(const MfmaArgs &a, const MItem &it,
                                                  f32x16m (&acc)[kMRB][NQB], int row0,
                                                  const float *ssc, int t) {
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int c = lane & 31, h = lane >> 5;
  const int lrow = wv * 32 * kMRB + 4 * h;
  const int lim0 = (int)a.N - row0 - lrow;
  const float *ssc_lane = FP8 ? ssc + lrow : nullptr;
  pin_acc(acc);
  finish_scores<FP8>(acc, ssc_lane, lim0);
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) {
    float m = -__builtin_inff();
#pragma unroll
    for (int rb = 0; rb < kMRB; ++rb)
#pragma unroll
      for (int i = 0; i < 16; ++i) m = fmaxf(m, acc[rb][qb][i]);
    const int ql = qb * 32 + c;
    if (ql < it.qvalid)
      a.lmax[(((int64_t)(it.qbase + ql) * it.S + it.s) * it.T + t) * kMLanesQ + wv * 2 + h] =
          m > -__builtin_inff() ? ord_score(m) : 0u;
  }
}

// Top-k epilogue of one tile.  row0 = corpus row of the tile's first row;
// ssc = row scales of the tile (fp8).
template <bool FP8, bool LDS_LISTS, int NQB>
__device__ __forceinline__ void mtile_epilogue(const MLds &L, const MfmaArgs &a, const MItem &it,
                                               f32x16m (&acc)[kMRB][NQB],
                                               float (&thr_r)[kMQB], int &epoch, int row0,
                                               const float *ssc, const uint32_t *gt,
                                               bool first) {
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int c = lane & 31, h = lane >> 5;
  const float ninf = -__builtin_inff();
  const int lrow = wv * 32 * kMRB + 4 * h;   // this lane's first row in the tile
  const int lim0 = (int)a.N - row0 - lrow;
  const float *ssc_lane = FP8 ? ssc + lrow : nullptr;
  pin_acc(acc);
  // fp8: scores are accumulator x row scale.  Only an item's first tile
  // (warm-up) scales the accumulators in place; otherwise the screening and
  // the examined blocks multiply as they read.
  const int gpl = mwarm_groups(a.k);
  const bool scaled = FP8 && first && gpl > 0;
  if (scaled)
    finish_scores<FP8>(acc, ssc_lane, lim0);
  else
    mask_tail(acc, lim0);
  if (first && gpl > 0) {
    // warm-up threshold: the smallest of kMLanesQ * gpl group maxima (the
    // queue, which these minima alias, is empty at an item's first tile)
    bar_lds();
    switch (gpl) {
      case 1: warm_minima<kMVals / 1, NQB>(L, acc, wv, c, h); break;
      case 2: warm_minima<kMVals / 2, NQB>(L, acc, wv, c, h); break;
      case 4: warm_minima<kMVals / 4, NQB>(L, acc, wv, c, h); break;
      case 8: warm_minima<kMVals / 8, NQB>(L, acc, wv, c, h); break;
      case 16: warm_minima<kMVals / 16, NQB>(L, acc, wv, c, h); break;
      case 32: warm_minima<kMVals / 32, NQB>(L, acc, wv, c, h); break;
      default: warm_minima<1, NQB>(L, acc, wv, c, h); break;
    }
    bar_lds();
    if (tid < it.qvalid) {
      float th = L.warm[tid];
#pragma unroll
      for (int w = 1; w < kMW; ++w) th = fminf(th, L.warm[w * kMMQ + tid]);
      L.thr0[tid] = th;
      L.thr[tid] = th;
      publish_thr(L, a, it, tid, th);
    }
    bar_lds();
#pragma unroll
    for (int qb = 0; qb < kMQB; ++qb) thr_r[qb] = L.thr[qb * 32 + c];
  }

  // shared thresholds of this lane's queries (read when the tile's copies
  // started; a stale value is just a lower bound)
  float g_r[kMQB];
#pragma unroll
  for (int qb = 0; qb < kMQB; ++qb) {
    const uint32_t gq = gt[qb * 32 + c];
    g_r[qb] = gq ? unord_score(gq) : -__builtin_inff();
    thr_r[qb] = fmaxf(thr_r[qb], g_r[qb]);
  }
  // Screening: elig[qb] bit 16 rb + i marks score (rb, qb, i) of this lane
  // as still to be examined; a 16-score row block is eligible when its best
  // score reaches the query threshold.
  pin_acc(acc);
  uint64_t elig[NQB];
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) elig[qb] = 0ull;
#pragma unroll
  for (int rb = 0; rb < kMRB; ++rb) {
    float s16[16];
    row_scales<FP8>(s16, ssc_lane, rb, scaled);
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) {
      float m = ninf;
#pragma unroll
      for (int i = 0; i < 16; ++i) m = fmaxf(m, FP8 ? acc[rb][qb][i] * s16[i] : acc[rb][qb][i]);
      elig[qb] |= m >= thr_r[qb] ? 0xFFFFull << (16 * rb) : 0ull;
    }
  }
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb)
    if (qb * 32 + c >= it.qvalid) elig[qb] = 0ull;
  // Scores at or above the current threshold are appended to the per-query
  // LDS queues (atomics, no barrier).  Merges into the k-lists are deferred:
  // one barrier per tile checks whether some queue overflowed (its
  // candidates stay eligible) or is due for a merge; only then do the
  // threads of the queries merge, the thresholds rise, and the candidates
  // left over are examined again.  A queue is due when half full if the
  // lists are in LDS, and only when full if they are in global memory,
  // where a merge round (two barriers and climbs through global memory)
  // costs more than the candidates a later threshold rise would save.
  constexpr int qdue = LDS_LISTS ? kMQcap / 2 : kMQcap;
  for (;;) {
    bool ovf = false, full = false;
    pin_acc(acc);
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) {
      const int ql = qb * 32 + c;
      const float th = thr_r[qb];
      uint64_t fail = 0;
#pragma unroll
      for (int rb = 0; rb < kMRB; ++rb) {
        const uint32_t el = (uint32_t)(elig[qb] >> (16 * rb)) & 0xFFFFu;
        if (!__builtin_amdgcn_ballot_w64(el != 0)) continue;
        float v[16], s16[16];
        row_scales<FP8>(s16, ssc_lane, rb, scaled);
        uint32_t cand = 0;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          v[i] = FP8 ? acc[rb][qb][i] * s16[i] : acc[rb][qb][i];
          cand |= v[i] >= th ? 1u << i : 0u;
        }
        cand &= el;
        if (!__builtin_amdgcn_ballot_w64(cand != 0)) continue;
        // one atomic per lane and block reserves queue slots for all its
        // candidates; the ones past the queue's room stay eligible
        const int rowb = opaque(row0 + lrow + rb * 32);
        int slot = 0;
        if (cand) slot = atomicAdd(&L.qcount[ql], __builtin_popcount(cand));
        while (cand) {
          if (slot >= kMQcap) {
            fail |= (uint64_t)cand << (16 * rb);
            ovf = true;
            break;
          }
          const int jx = __builtin_ctz(cand);
          cand &= cand - 1u;
          // v[jx] by a tree of bitwise selects on the bits of jx (opaque
          // all-ones / zero masks: as plain selects, the compiler turns the
          // tree into an indexed load from scratch memory)
          uint32_t w8[8], w4[4];
          const uint32_t m0 = (uint32_t)opaque(-(jx & 1)), m1 = (uint32_t)opaque(-((jx >> 1) & 1));
          const uint32_t m2 = (uint32_t)opaque(-((jx >> 2) & 1)), m3 = (uint32_t)opaque(-(jx >> 3));
#pragma unroll
          for (int i = 0; i < 8; ++i)
            w8[i] = (__float_as_uint(v[2 * i]) & ~m0) | (__float_as_uint(v[2 * i + 1]) & m0);
#pragma unroll
          for (int i = 0; i < 4; ++i) w4[i] = (w8[2 * i] & ~m1) | (w8[2 * i + 1] & m1);
          const uint32_t w2a = (w4[0] & ~m2) | (w4[1] & m2), w2b = (w4[2] & ~m2) | (w4[3] & m2);
          const float sc = __uint_as_float((w2a & ~m3) | (w2b & m3));
          full |= slot + 1 >= qdue;
          L.queue[ql * kMQcap + slot] = make_key(sc, (uint32_t)(rowb + 8 * (jx >> 2) + (jx & 3)));
          ++slot;
        }
      }
      elig[qb] = fail;
    }
    if (__builtin_amdgcn_ballot_w64(ovf) && lane == 0) L.flags[1] = epoch;
    if (__builtin_amdgcn_ballot_w64(full) && lane == 0) L.flags[2] = epoch;
    bar_lds();
    const bool again = L.flags[1] == epoch;
    if (!again && L.flags[2] != epoch) {   // no queue needs a merge yet
      ++epoch;
      break;
    }
    if (tid < it.qvalid) merge_queue<LDS_LISTS>(L, a, it, tid);
    bar_lds();
#pragma unroll
    for (int qb = 0; qb < kMQB; ++qb) thr_r[qb] = fmaxf(L.thr[qb * 32 + c], g_r[qb]);
    ++epoch;
    if (!again) break;
  }
}

// One work item (a query tile against one corpus slice) whose queries fill
// NQB of the tile's 32-query blocks: the fragment reads, the matrix-core
// steps and the epilogue skip the blocks past the item's queries (few
// distinct queries).  The copies are those of a full
// tile (the query rows past the item's queries read as zeros).
template <bool FP8, bool LDS_LISTS, bool SEED, int NQB>
__device__ __forceinline__ void run_item(const MfmaArgs &a, const MLds &L, const Split &sp,
                                         int64_t nu, int w, int &epoch) {
  using G = Geo<FP8>;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int c = lane & 31, h = lane >> 5;
  const int N = (int)a.N, d = (int)a.d;
  const int nch = (d + kMKC - 1) / kMKC;
  const float ninf = -__builtin_inff();
  // (the per-lane copy offsets are recomputed at each copy from the lane id,
  // a few VALU operations, rather than held in registers across the loop)
  {
    MItem it;
    const int qt = w % (int)sp.qtiles;
    it.s = w / (int)sp.qtiles;
    it.S = sp.S;
    it.T = seed_tiles(a.k, sp.ntiles, sp.S);
    const int s0 = (int)((int64_t)it.s * sp.ntiles / sp.S);
    const int s1 = (int)((int64_t)(it.s + 1) * sp.ntiles / sp.S);
    const int t0 = s0;
    const int t1 = SEED ? s0 + (s1 - s0 < it.T ? s1 - s0 : it.T) : s1;
    it.qbase = qt * kMMQ;
    it.qvalid = (int)(nu - it.qbase < kMMQ ? nu - it.qbase : kMMQ);
    const int ntl = t1 - t0;
    const int T = ntl * nch;
    if constexpr (SEED) {
      if (it.s % seed_stride(it.S) != 0) {   // not sampled: no lane maxima
        const int per = it.T * kMLanesQ;
        for (int e = tid; e < it.qvalid * per; e += kMT) {
          const int qq = e / per, r = e - qq * per;
          a.lmax[((int64_t)(it.qbase + qq) * it.S + it.s) * per + r] = 0u;
        }
        return;
      }
    }

    // per-item state
    if (tid < kMMQ) {
      L.qcount[tid] = 0;
      L.thr0[tid] = ninf;
      L.thr[tid] = ninf;
      L.lmin[tid] = 0ull;
      L.pub[tid] = 0u;
      if (tid < it.qvalid && !SEED) {
        // (items of the first round start before any item has finished)
        if (w >= a.grid) {
          const uint32_t b =
              level_bound(a.lvl + (int64_t)(it.qbase + tid) * kLvl * it.S, (int)it.S);
          if (b) {
            atomicMax(a.gthr + it.qbase + tid, b);
            L.pub[tid] = b;
          }
        }
        if (LDS_LISTS) {
          for (int j = 0; j < a.k; ++j) L.lists[tid * a.k + j] = 0ull;
        } else {
          uint64_t *l = a.part + ((int64_t)(it.qbase + tid) * it.S + it.s) * a.k;
          for (int j = 0; j < a.k - kMTail; ++j) l[j] = 0ull;
          for (int j = 0; j < kMTail; ++j) L.tail[tid * kMTail + j] = 0ull;
        }
      }
    }
    float thr_r[kMQB];   // (read from L.thr after the prologue barrier)

    // the query tile's rows in the tiled order of tile_queries_kernel: stage
    // s of the tile is the 16 KiB block s, already in LDS order
    const i32x4m qrs =
        make_rsrc((const unsigned char *)a.q + (int64_t)(it.qbase / kMMQ) * nch * G::bbytes,
                  (uint32_t)(nch * G::bbytes));

    // copy stream: next chunk to issue.  A chunk is copied in two parts:
    // issue_a copies the corpus rows of this wave (the only wave that reads
    // them) and issue_b the wave's share of the query rows, the tile's shared
    // thresholds and row scales, and advances the stream.  issue_a of a
    // chunk always precedes its issue_b.
    int i_tl = 0, i_kc = 0, i_slot = 0, i_sc = 0, i_gt = 0, i_left = T;
    struct CopyA {
      i32x4m rs;
      uint32_t lds, voff, voff1;
    };
    auto prep_a = [&]() __attribute__((always_inline)) {
      CopyA ca;
      unsigned char *st = L.ring + i_slot * G::stage;
      const int ln = opaque(lane);
      constexpr int PA = G::apieces;
      const int wvs = __builtin_amdgcn_readfirstlane(wv);
      ca.lds = (uint32_t)(uintptr_t)st + wvs * G::adma * 1024;
      if (a.tiled) {
        // the tile's stages are consecutive blocks already in LDS order: this
        // wave's copies read adma consecutive KiB of the stage's block
        const uint32_t tb = (uint32_t)(nch * G::abytes);
        ca.rs = make_rsrc((const unsigned char *)a.corpus + (int64_t)(t0 + i_tl) * tb, tb);
        ca.voff = (uint32_t)((i_kc / kMKC) * G::abytes + wvs * G::adma * 1024 + ln * 16);
        ca.voff1 = ca.voff;
        return ca;
      }
      const int row0 = (t0 + i_tl) * kMNC;
      const int rows = N - row0 < kMNC ? N - row0 : kMNC;
      ca.rs = make_rsrc((const unsigned char *)a.corpus + (int64_t)row0 * d * G::esz,
                        (uint32_t)(rows * d * G::esz));
      const int arow0 = wvs * G::adma * (64 / PA) + ln / PA;
      ca.voff = (uint32_t)(arow0 * d * G::esz + swz_slot<PA>(ln % PA, ln / PA) * 16 + i_kc * G::esz);
      // the swizzle depends on the row mod 16: a bf16 copy holds 8 rows, so odd
      // copies hold rows 8..15 mod 16 (an fp8 copy holds 16 rows: one pattern)
      ca.voff1 = (uint32_t)(arow0 * d * G::esz +
                            swz_slot<PA>(ln % PA, (64 / PA) % 16 + ln / PA) * 16 + i_kc * G::esz);
      return ca;
    };
    auto issue_a_j = [&](const CopyA &ca, int j) __attribute__((always_inline)) {
      constexpr int PA = G::apieces;
      const uint32_t jstep = a.tiled ? 1024u : (uint32_t)((64 / PA) * d * G::esz);
      dma16s(ca.rs, ca.lds + j * 1024, ((j & 1) ? ca.voff1 : ca.voff) + (uint32_t)j * jstep);
    };
    auto issue_a = [&]() __attribute__((always_inline)) {
      if (i_left <= 0) return;
      const CopyA ca = prep_a();
#pragma unroll
      for (int j = 0; j < G::adma; ++j) issue_a_j(ca, j);
    };
    struct CopyB {
      uint32_t lds, voff;
    };
    // query part of the next chunk: this wave's bdma consecutive KiB of the
    // stage's block (queries past n_u and columns past d are zeros there);
    // once the stream has ended, zeros through an offset past the range
    auto prep_b = [&]() __attribute__((always_inline)) {
      CopyB cb;
      const int ln = opaque(lane);
      const int wvs = __builtin_amdgcn_readfirstlane(wv);
      cb.voff = i_left > 0
                    ? (uint32_t)((i_kc / kMKC) * G::bbytes + wvs * G::bdma * 1024 + ln * 16)
                    : 0x80000000u;
      cb.lds = (uint32_t)(uintptr_t)(L.ring + i_slot * G::stage + G::abytes) + wvs * G::bdma * 1024;
      return cb;
    };
    auto issue_b_j = [&](const CopyB &cb, int j) __attribute__((always_inline)) {
      dma16s(qrs, cb.lds + j * 1024, cb.voff + (uint32_t)(j * 1024));
    };
    auto extras_advance = [&]() __attribute__((always_inline)) {
      if (i_left <= 0) return;
      const int ln = opaque(lane);
      if (i_kc == 0) {
        // shared thresholds of the query tile, entries [32 wv, 32 wv + 64)
        const i32x4m grs = make_rsrc(a.gthr + it.qbase, (uint32_t)(it.qvalid * 4));
        dma4(grs, L.gtl + i_gt * kMGts + 32 * wv, (uint32_t)((32 * wv + ln) * 4));
        i_gt = i_gt + 1 == G::ngt ? 0 : i_gt + 1;
      }
      if constexpr (FP8) {
        if (i_kc == 0) {
          // rows [kMRowsW * wv, + 128) of the tile: the wave's own rows and an
          // overlap with the next wave's (same values, same place)
          const int row0 = (t0 + i_tl) * kMNC;
          const int rows = N - row0 < kMNC ? N - row0 : kMNC;
          const i32x4m srs = make_rsrc(a.scale + row0, (uint32_t)(rows * 4));
#pragma unroll
          for (int j = 0; j < 2; ++j)
            dma4(srs, L.sscale + i_sc * kMSS + wv * kMRowsW + j * 64,
                 (uint32_t)((wv * kMRowsW + j * 64 + ln) * 4));
          i_sc = i_sc + 1 == G::nsc ? 0 : i_sc + 1;
        }
      }
      i_kc += kMKC;
      if (i_kc >= d) {
        i_kc = 0;
        ++i_tl;
      }
      i_slot = i_slot + 1 == G::ns ? 0 : i_slot + 1;
      --i_left;
    };
    auto issue_b = [&]() __attribute__((always_inline)) {
      const CopyB cb = prep_b();
#pragma unroll
      for (int j = 0; j < G::bdma; ++j) issue_b_j(cb, j);
      extras_advance();
    };
    // Vector-memory operations issued after the query part of chunk y, up
    // to the corpus part of chunk z (only z's corpus part is issued yet).
    // Tile-first extras are not counted: waiting for fewer outstanding
    // operations only waits longer.
    auto younger_ops = [&](int y, int z) __attribute__((always_inline)) {
      int n = 0;
      for (int x = y + 1; x <= z && x < T; ++x) n += x < z ? G::ldma : G::adma;
      return n;
    };

#pragma unroll
    for (int j = 0; j < G::ns; ++j) {
      issue_a();
      issue_b();
    }
    // chunk 0 landed (chunks 1 .. ns-1 are younger)
    wait_vm(((T < G::ns ? T : G::ns) - 1) * G::ldma);
    bar_lds();

#pragma unroll
    for (int qb = 0; qb < kMQB; ++qb) thr_r[qb] = L.thr[qb * 32 + c];
    f32x16m acc[kMRB][NQB];
    Frag<FP8, NQB> f0, f1;
    read_frags<FP8>(f0, L.ring, wv, c, h, 0);
    int r_slot = 0, e_sc = 0, e_gt = 0, g = 0;

    // One stage: two halves of two MFMA steps each.  Once this wave's reads
    // of the stage's slot are complete (after step 0) it refills its own
    // corpus rows there with stage g+ns; no other wave reads them, so no
    // barrier is needed, and these copies (three quarters of the bytes)
    // get about half a stage more to arrive.  Before step 3 the wave waits
    // for stage g+1, the barrier lets every wave's copies of it be read and
    // lets the query rows of the slot be refilled, and the next stage's
    // first fragments are read, so that reads overlap the last MFMAs.
    // (Moving the whole copy earlier costs a second barrier per stage, which
    // was slower: the loop is bound by the matrix cores sharing the CU with
    // the LDS reads more than by copy latency.)
    auto stage = [&](auto first_c, bool rd) __attribute__((always_inline)) {
      constexpr bool FIRST = decltype(first_c)::value;
      constexpr int NR = Frag<FP8, NQB>::nreads;
      const unsigned char *cur = L.ring + r_slot * G::stage;
      const int ln1 = opaque(lane);
      mfma_step_il<FP8, FIRST, NR>(acc, f0, 0, [&](int k) __attribute__((always_inline)) {
        read_frag_piece<FP8>(f1, cur, wv, ln1 & 31, ln1 >> 5, 1, k);
      });
      {
        __builtin_amdgcn_sched_barrier(0);
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __builtin_amdgcn_sched_barrier(0);
        CopyA ca = prep_a();   // this wave's corpus rows of stage g+ns
        if (i_left <= 0) ca.rs.z = 0;
        mfma_step_il<FP8, false, G::adma>(acc, f0, 1, [&](int k) __attribute__((always_inline)) {
          issue_a_j(ca, k);
        });
      }
      mfma_step<FP8, false>(acc, f1, 0);
      r_slot = r_slot + 1 == G::ns ? 0 : r_slot + 1;
      // stage g+1 landed (after the last stage: all copies landed):
      // younger are the parts of stages g+2 .. g+ns issued so far
      wait_vm(younger_ops(g + 1, g + G::ns));
      bar_lds();
      pin_step1<FP8>(f1);
      const CopyB cb = prep_b();   // query rows of stage g+ns into the slot stage g used
      const unsigned char *nxt = L.ring + r_slot * G::stage;
      const int ln0 = opaque(lane);
      mfma_step_il<FP8, false, G::bdma + NR>(acc, f1, 1, [&](int k) __attribute__((always_inline)) {
        if (k < G::bdma)
          issue_b_j(cb, k);
        else if (rd)
          read_frag_piece<FP8>(f0, nxt, wv, ln0 & 31, ln0 >> 5, 0, k - G::bdma);
      });
      extras_advance();
      ++g;
    };
    // (the first stage of a tile starts the accumulators from zero; its call
    // is peeled so that the previous tile's accumulators are dead here.  The
    // last stage of a tile leaves the next fragments in LDS: the epilogue runs
    // with only the accumulators live, and f0 is refilled after it.)
    for (int tl = 0; tl < ntl; ++tl) {
      stage(std::true_type{}, nch > 1);
      for (int j = 1; j < nch; ++j) stage(std::false_type{}, j + 1 < nch);
      if constexpr (SEED)
        mtile_lane_maxima<FP8>(a, it, acc, (t0 + tl) * kMNC,
                               FP8 ? L.sscale + e_sc * kMSS : nullptr, tl);
      else
        mtile_epilogue<FP8, LDS_LISTS>(L, a, it, acc, thr_r, epoch, (t0 + tl) * kMNC,
                                       FP8 ? L.sscale + e_sc * kMSS : nullptr,
                                       L.gtl + e_gt * kMGts, tl == 0);
      if constexpr (FP8) e_sc = e_sc + 1 == G::nsc ? 0 : e_sc + 1;
      e_gt = e_gt + 1 == G::ngt ? 0 : e_gt + 1;
      read_frags<FP8>(f0, L.ring + r_slot * G::stage, wv, c, h, 0);
    }

    if constexpr (SEED) {   // sampled tiles this slice does not have: no value
      const int st = it.T;
      for (int e = tid; e < it.qvalid * (st - ntl) * kMLanesQ; e += kMT) {
        const int q = e / ((st - ntl) * kMLanesQ), r = e % ((st - ntl) * kMLanesQ);
        a.lmax[(((int64_t)(it.qbase + q) * it.S + it.s) * st + ntl) * kMLanesQ + r] = 0u;
      }
    }
    // merge what is still queued, then flush the LDS lists of this item
    if constexpr (!SEED) {
      bar_lds();
      if (tid < it.qvalid) {
        merge_queue<LDS_LISTS>(L, a, it, tid);
        // this slice's order statistics for the items that start later
        const uint64_t mn = L.lmin[tid];
        const int fill = (mn >> 32) ? a.k : (int)mn;
        const uint64_t *gl = a.part + ((int64_t)(it.qbase + tid) * it.S + it.s) * a.k;
        uint32_t *lv = a.lvl + (int64_t)(it.qbase + tid) * kLvl * it.S + it.s;
        for (int l = 0; l < kLvl; ++l) {
          const int p = opaque(((a.k + (1 << l) - 1) >> l) - 1);   // ceil(k / 2^l) - 1
          if (p < fill) {
            uint64_t key;
            if (LDS_LISTS)
              key = L.lists[tid * a.k + p];
            else if (p >= a.k - kMTail)
              key = L.tail[tid * kMTail + p - (a.k - kMTail)];
            else
              key = gl[p];
            __hip_atomic_store(lv + l * it.S, (uint32_t)(key >> 32), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
          }
        }
      }
    }
    if (LDS_LISTS && !SEED) {
      bar_lds();
      const int tot = it.qvalid * a.k;
      for (int t = tid; t < tot; t += kMT) {
        const int q = t / a.k, j = t - q * a.k;
        a.part[((int64_t)(it.qbase + q) * it.S + it.s) * a.k + j] = L.lists[t];
      }
    }
    if (!LDS_LISTS && !SEED) {
      bar_lds();
      const int tot = it.qvalid * kMTail;
      for (int t = tid; t < tot; t += kMT) {
        const int q = t / kMTail, j = t - q * kMTail;
        a.part[((int64_t)(it.qbase + q) * it.S + it.s) * a.k + a.k - kMTail + j] = L.tail[t];
      }
    }
    wait_vm(0);
    bar_lds();
  }
}

template <bool FP8, bool LDS_LISTS, bool SEED>
__global__ __launch_bounds__(kMT, 1) void score_mfma_dma(MfmaArgs a) {
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  const MLds L = carve_mlds<FP8, LDS_LISTS>(smem, a.k);
  const int64_t nu = read_nu(a.n_unique, a.n_unique_dev, a.cap);
  int64_t smax = kMSplitMaxSK / a.k;
  const Split sp = make_split(nu, a.N, kMMQ, kMNC, a.grid, smax < 1 ? 1 : smax);
  const int items = (int)(sp.qtiles * sp.S);
  if (threadIdx.x < 4) L.flags[threadIdx.x] = 0;
  int epoch = 1;
  for (int w = logical_wg(a.grid); w < items; w += a.grid) {
    // Queries of the item's tile (at least one: the tiles cover n_u).  With
    // several query tiles, the items of one corpus slice run on neighbouring
    // workgroups of one XCD and share its L2 only while they run at the same
    // pace, so every item then runs as a full tile; a single (partial) tile
    // skips its empty query blocks.
    const int64_t qv = sp.qtiles > 1 ? kMMQ : nu;
    if (qv > 96)
      run_item<FP8, LDS_LISTS, SEED, 4>(a, L, sp, nu, w, epoch);
    else if (qv > 64)
      run_item<FP8, LDS_LISTS, SEED, 3>(a, L, sp, nu, w, epoch);
    else if (qv > 32)
      run_item<FP8, LDS_LISTS, SEED, 2>(a, L, sp, nu, w, epoch);
    else
      run_item<FP8, LDS_LISTS, SEED, 1>(a, L, sp, nu, w, epoch);
  }
}

// ---------------------------------------------------------------- host side

int persistent_grid(bool mfma);

// Score workspace of the matrix-core path: [shared thresholds, cap x u32]
// (rounded to 256 bytes) followed by the partial lists.
size_t mfma_thr_bytes(int64_t cap) { return ((size_t)cap * 4 + 255) & ~(size_t)255; }

// worst case over n_u in [1, cap] and grids up to grid_max of n_u * S * f(k),
// f(k) = per_slice bytes, times the seed pass's tiles per slice if seed.
// It takes up to (cap / 128) x 64 splits, and every score call lays out its
// workspace with it, so results are kept for the few shapes a process uses
// (on a window of a few hundred queries the loops cost tens of microseconds,
// on the launch path).
struct SplitWorstMemo {
  int64_t cap, N;
  int k, grid_max;
  size_t per_slice;
  bool seed, valid;
  size_t bytes;
};
static std::mutex g_split_memo_mu;
static SplitWorstMemo g_split_memo[16];
static unsigned g_split_memo_next = 0;

static size_t mfma_split_worst(int64_t cap, int64_t N, int k, int grid_max, size_t per_slice,
                               bool seed = false) {
  {
    std::lock_guard<std::mutex> lock(g_split_memo_mu);
    for (const SplitWorstMemo &m : g_split_memo)
      if (m.valid && m.cap == cap && m.N == N && m.k == k && m.grid_max == grid_max &&
          m.per_slice == per_slice && m.seed == seed)
        return m.bytes;
  }
  size_t best = 0;
  const int64_t qtmax = (cap + kMMQ - 1) / kMMQ;
  int64_t smax = kMSplitMaxSK / k;
  if (smax < 1) smax = 1;
  for (int64_t qt = 1; qt <= qtmax; ++qt) {
    const int64_t nu = qt * kMMQ < cap ? qt * kMMQ : cap;
    for (int64_t g = 8; g <= grid_max; g += 8) {
      const Split sp = make_split(nu, N, kMMQ, kMNC, g, smax);
      const size_t b = (size_t)nu * (size_t)sp.S * per_slice *
                       (seed ? (size_t)seed_tiles(k, sp.ntiles, sp.S) : 1u);
      if (b > best) best = b;
    }
  }
  best = (best + 255) & ~(size_t)255;
  std::lock_guard<std::mutex> lock(g_split_memo_mu);
  g_split_memo[g_split_memo_next++ % 16] = {cap, N, k, grid_max, per_slice, seed, true, best};
  return best;
}

// Score workspace of the matrix-core path: [shared thresholds, cap x u32 |
// seed-pass lane maxima, n_u x S x T x 8 u32 | order statistics of finished
// items, n_u x kLvl x S u32 | partial lists, n_u x S x k keys],
// each rounded to 256 bytes.
size_t mfma_lmax_bytes(int64_t cap, int64_t N, int k, int grid_max) {
  return mfma_split_worst(cap, N, k, grid_max, (size_t)kMLanesQ * 4, true);
}

// published order statistics, n_u x S x kLvl u32
static size_t mfma_lvl_bytes(int64_t cap, int64_t N, int k, int grid_max) {
  return mfma_split_worst(cap, N, k, grid_max, (size_t)kLvl * 4);
}

size_t mfma_partial_bytes(int64_t cap, int64_t N, int k, int grid_max) {
  return mfma_thr_bytes(cap) + mfma_lmax_bytes(cap, N, k, grid_max) +
         mfma_lvl_bytes(cap, N, k, grid_max) +
         mfma_split_worst(cap, N, k, grid_max, (size_t)k * 8);
}

// Offset of the partial lists in the score workspace.
size_t mfma_part_offset(int64_t cap, int64_t N, int k, int grid_max) {
  return mfma_thr_bytes(cap) + mfma_lmax_bytes(cap, N, k, grid_max) +
         mfma_lvl_bytes(cap, N, k, grid_max);
}

void mfma_split_params(int *mq, int *nc, int64_t *smax, int k) {
  *mq = kMMQ;
  *nc = kMNC;
  int64_t s = kMSplitMaxSK / k;
  *smax = s < 1 ? 1 : s;
}

template <typename K>
static hipError_t launch_mfma(K kern, int grid, int lds, const MfmaArgs &a, hipStream_t st) {
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(grid), dim3(kMT), lds, st, a);
  return hipGetLastError();
}

// Threshold seed per distinct query: the k-th largest of its lane maxima
// from the seed pass (at most kSeedMax of them), written to gthr, which it
// thereby (re)starts for the call: 0, no threshold, where there is no seed.
// The seed pass reads gthr only with its copies and never uses the values.
// Radix
// select on the 32-bit ordered scores, 8 bits per pass: a pass counts the
// values that carry the digits chosen so far by their next digit, and keeps
// the largest digit whose count of values at or above it reaches the rank
// still sought.
constexpr int kSeedThreads = 256;
__global__ __launch_bounds__(kSeedThreads) void mfma_seed_kernel(
    const uint32_t *__restrict__ lmax, int64_t n_unique, const int64_t *__restrict__ nu_dev,
    int64_t cap, int64_t N, int k, int64_t smax, int grid, uint32_t *__restrict__ gthr,
    uint32_t *__restrict__ lvl) {
  __shared__ uint32_t vals[kSeedMax];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t sel[2];   // chosen digit, values above it
  const int64_t nu = read_nu(n_unique, nu_dev, cap);
  const Split sp = make_split(nu, N, kMMQ, kMNC, grid, smax);
  const int64_t per = sp.S * kMLanesQ * seed_tiles(k, sp.ntiles, sp.S);
  const int n = (int)(per < kSeedMax ? per : kSeedMax);
  const int tid = threadIdx.x;
  // no item of this call has finished yet: no published order statistics
  for (int64_t e = (int64_t)blockIdx.x * kSeedThreads + tid; e < nu * kLvl * sp.S;
       e += (int64_t)gridDim.x * kSeedThreads)
    lvl[e] = 0u;
  if (n < k) {   // fewer lane maxima than k: no seed
    for (int64_t q = (int64_t)blockIdx.x * kSeedThreads + tid; q < nu;
         q += (int64_t)gridDim.x * kSeedThreads)
      gthr[q] = 0u;
    return;
  }
  for (int64_t q = blockIdx.x; q < nu; q += gridDim.x) {
    const uint32_t *src = lmax + q * per;
    for (int i = tid; i < n; i += kSeedThreads) vals[i] = src[i];
    uint32_t prefix = 0u, pmask = 0u;
    int kk = k;   // rank sought among the values that carry prefix
    for (int shift = 24; shift >= 0; shift -= 8) {
      hist[tid] = 0u;
      __syncthreads();
      for (int i = tid; i < n; i += kSeedThreads) {
        const uint32_t v = vals[i];
        if ((v & pmask) == prefix) atomicAdd(&hist[(v >> shift) & 0xFFu], 1u);
      }
      __syncthreads();
      if (tid < kWave) {
        // lane l holds digits 255 - 4l - j (j = 0..3), largest first; an
        // exclusive scan over lanes counts the values above its digits
        uint32_t c[4], sum = 0u;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          c[j] = hist[255 - 4 * tid - j];
          sum += c[j];
        }
        uint32_t incl = sum;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
          const uint32_t t = __shfl_up(incl, o);
          if (tid >= o) incl += t;
        }
        uint32_t above = incl - sum;
        if (above < (uint32_t)kk && (uint32_t)kk <= incl) {
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            if (above + c[j] >= (uint32_t)kk) {
              sel[0] = 255u - 4u * tid - j;
              sel[1] = above;
              break;
            }
            above += c[j];
          }
        }
      }
      __syncthreads();
      prefix |= sel[0] << shift;
      pmask |= 0xFFu << shift;
      kk -= (int)sel[1];
      // (hist was last read before the barrier above; sel is rewritten only
      // after the next pass's counting barrier)
    }
    if (tid == 0) gthr[q] = prefix;
    __syncthreads();
  }
}

// Tiled corpus layout.  Tile t (corpus rows [384 t, 384 t + 384)) and stage s
// (columns [64 s, 64 s + 64)) form one block of Geo::abytes bytes at
// (t * nch + s) * Geo::abytes, nch = ceil(d / 64): the stage exactly as the
// copies place it in LDS, row r of the tile at r * Geo::arow with its 16-byte
// pieces in the swizzled slots the fragment reads expect (slot x of row r holds
// piece swz_slot(x, r)).  Rows past N and columns past d are zeros.  The score
// kernel then copies each wave's share of a stage as consecutive KiB instead of
// 8 (bf16) or 16 (fp8) row pieces per copy.
template <bool FP8>
__global__ __launch_bounds__(256) void tile_corpus_kernel(const unsigned char *__restrict__ src,
                                                          int64_t N, int64_t d, int nch,
                                                          int64_t npieces,
                                                          uint4 *__restrict__ dst) {
  using G = Geo<FP8>;
  constexpr int PA = G::apieces;
  constexpr int per_stage = G::abytes / 16;
  for (int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x; p < npieces;
       p += (int64_t)gridDim.x * 256) {
    const int64_t blk = p / per_stage;
    const int in = (int)(p - blk * per_stage);
    const int64_t t = blk / nch;
    const int s = (int)(blk - t * nch);
    const int r = in / PA;
    const int piece = swz_slot<PA>(in % PA, r);   // (an XOR: slot -> piece)
    const int64_t row = t * kMNC + r;
    const int64_t col = (int64_t)s * kMKC + piece * (16 / G::esz);
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (row < N && col < d)
      v = *reinterpret_cast<const uint4 *>(src + (row * d + col) * G::esz);
    dst[p] = v;
  }
}

// The distinct queries in the same order, per query tile: tile u (queries
// [128 u, 128 u + 128)) and stage s form the 16 KiB block u * nch + s, row r
// of the tile at r * 128 bytes with its pieces in the swizzled slots; queries
// past n_u and columns past d are zeros.  Written into the score workspace at
// the start of every score call (n_u * d * 2 bytes read, the tiles' bytes
// written), so that the score kernel's query copies read consecutive KiB too.
__global__ __launch_bounds__(256) void tile_queries_kernel(
    const unsigned char *__restrict__ q, int64_t n_unique, const int64_t *__restrict__ nu_dev,
    int64_t cap, int64_t d, int nch, uint4 *__restrict__ dst) {
  constexpr int PB = Geo<false>::bpieces;
  constexpr int per_stage = Geo<false>::bbytes / 16;
  const int64_t nu = read_nu(n_unique, nu_dev, cap);
  const int64_t npieces = (nu + kMMQ - 1) / kMMQ * nch * per_stage;
  for (int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x; p < npieces;
       p += (int64_t)gridDim.x * 256) {
    const int64_t blk = p / per_stage;
    const int in = (int)(p - blk * per_stage);
    const int64_t u = blk / nch;
    const int s = (int)(blk - u * nch);
    const int r = in / PB;
    const int piece = swz_slot<PB>(in % PB, r);
    const int64_t row = u * kMMQ + r;
    const int64_t col = (int64_t)s * kMKC + piece * 8;
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (row < nu && col < d) v = *reinterpret_cast<const uint4 *>(q + (row * d + col) * 2);
    dst[p] = v;
  }
}

// Bytes of the tiled queries for up to cap distinct queries.
size_t mfma_qtile_bytes(int64_t cap, int64_t d) {
  return (size_t)((cap + kMMQ - 1) / kMMQ) * (size_t)((d + kMKC - 1) / kMKC) * Geo<false>::bbytes;
}

// Offset of the tiled queries in the score workspace (after the partial lists).
size_t mfma_qtile_offset(int64_t cap, int64_t N, int k, int grid_max) {
  return (mfma_partial_bytes(cap, N, k, grid_max) + 255) & ~(size_t)255;
}

size_t mfma_tiled_bytes(int64_t N, int64_t d, bool fp8) {
  const int64_t tiles = (N + kMNC - 1) / kMNC, nch = (d + kMKC - 1) / kMKC;
  return (size_t)(tiles * nch) * (size_t)(fp8 ? Geo<true>::abytes : Geo<false>::abytes);
}

hipError_t launch_tile_corpus(const void *corpus, int64_t N, int64_t d, bool fp8, void *tiled,
                              hipStream_t st) {
  const int64_t npieces = (int64_t)(mfma_tiled_bytes(N, d, fp8) / 16);
  if (npieces == 0) return hipSuccess;
  const int nch = (int)((d + kMKC - 1) / kMKC);
  const int64_t want = (npieces + 255) / 256;
  const unsigned blocks = (unsigned)(want < 8192 ? want : 8192);
  if (fp8)
    hipLaunchKernelGGL(tile_corpus_kernel<true>, dim3(blocks), dim3(256), 0, st,
                       (const unsigned char *)corpus, N, d, nch, npieces, (uint4 *)tiled);
  else
    hipLaunchKernelGGL(tile_corpus_kernel<false>, dim3(blocks), dim3(256), 0, st,
                       (const unsigned char *)corpus, N, d, nch, npieces, (uint4 *)tiled);
  return hipGetLastError();
}

hipError_t launch_score_mfma(const void *q, const void *corpus, const float *scale, int64_t N,
                             int64_t d, int k, int64_t n_unique, const int64_t *nu_dev,
                             int64_t cap, bool fp8, bool tiled, void *ws, hipStream_t st) {
  // shared thresholds: (re)started by the seed selection on every call
  uint32_t *gthr = (uint32_t *)ws;
  uint32_t *lmax = (uint32_t *)((unsigned char *)ws + mfma_thr_bytes(cap));
  uint32_t *lvl = (uint32_t *)((unsigned char *)ws + mfma_thr_bytes(cap) +
                               mfma_lmax_bytes(cap, N, k, kMGridMax));
  void *part = (unsigned char *)ws + mfma_part_offset(cap, N, k, kMGridMax);
  void *qt = (unsigned char *)ws + mfma_qtile_offset(cap, N, k, kMGridMax);
  if (cap > 0) {
    const int nch = (int)((d + kMKC - 1) / kMKC);
    const int64_t want = (int64_t)(mfma_qtile_bytes(cap, d) / 16 + 255) / 256;
    const unsigned blocks = (unsigned)(want < 2048 ? want : 2048);
    hipLaunchKernelGGL(tile_queries_kernel, dim3(blocks), dim3(256), 0, st,
                       (const unsigned char *)q, n_unique, nu_dev, cap, d, nch, (uint4 *)qt);
    hipError_t e0 = hipGetLastError();
    if (e0 != hipSuccess) return e0;
  }
  MfmaArgs a;
  a.q = qt;
  a.corpus = corpus;
  a.scale = scale;
  a.N = N;
  a.d = d;
  a.k = k;
  a.n_unique = n_unique;
  a.n_unique_dev = nu_dev;
  a.cap = cap;
  a.part = (uint64_t *)part;
  a.gthr = gthr;
  a.lmax = lmax;
  a.lvl = lvl;
  a.grid = persistent_grid(true);
  a.tiled = tiled ? 1 : 0;
  // k-lists in LDS when they fit beside the ring
  const bool ll = mfma_lds_bytes(fp8, true, k) <= kMLdsMax;
  const int lds = mfma_lds_bytes(fp8, ll, k);
  const int lds_seed = mfma_lds_bytes(fp8, false, k);
  auto run = [&](bool seed) {
    if (seed) return fp8 ? launch_mfma(score_mfma_dma<true, false, true>, a.grid, lds_seed, a, st)
                         : launch_mfma(score_mfma_dma<false, false, true>, a.grid, lds_seed, a, st);
    if (fp8) return ll ? launch_mfma(score_mfma_dma<true, true, false>, a.grid, lds, a, st)
                       : launch_mfma(score_mfma_dma<true, false, false>, a.grid, lds, a, st);
    return ll ? launch_mfma(score_mfma_dma<false, true, false>, a.grid, lds, a, st)
              : launch_mfma(score_mfma_dma<false, false, false>, a.grid, lds, a, st);
  };
  // Seed pass: score the first T tiles of every sampled slice (all slices, or
  // one in seed_stride(S)) and keep only lane maxima; their k-th largest per
  // query (a lower bound of the query's k-th best over the corpus, taken over
  // a sample of tiles spread over it)
  // seeds the shared thresholds.  The main pass then scores every tile with
  // lists that stay nearly untouched from the first tile on.
  hipError_t e = run(true);
  if (e != hipSuccess) return e;
  if (cap > 0) {
    int64_t smax = kMSplitMaxSK / k;
    if (smax < 1) smax = 1;
    const int64_t want = n_unique >= 0 ? n_unique : cap;
    const int64_t blocks = want < 4 * (int64_t)a.grid ? want : 4 * (int64_t)a.grid;
    if (blocks > 0) {
      hipLaunchKernelGGL(mfma_seed_kernel, dim3((unsigned)blocks), dim3(kSeedThreads), 0, st,
                         a.lmax, n_unique, nu_dev, cap, N, k, smax, a.grid, gthr, a.lvl);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
  }
  return run(false);
}

}  // namespace hs
