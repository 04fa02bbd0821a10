// Node semantic signatures on the device.
//
// HeraSys Eq. 2: a node's signature hashes its operator type tau_v, the
// parameters that affect its result Theta_p, the input data D_in that fixes
// its output (for retrieval and embedding nodes, the normalised query text or
// the chunk content) and the ordered signatures of its predecessors.  The
// prototype hashes with SHA-256 (Sec. 4.1, testbed).  The message of node v is
// the length-prefixed concatenation (all integers little-endian)
//
//   le32(tau_v) | le32(|Theta|) | Theta | le32(|D|) | D | le32(m) |
//   Sig(u_1) | ... | Sig(u_m)
//
// where D is the node's text, normalised or not, and Sig(u_j) are the 32-byte
// digests of the m predecessors in their given order.  The length prefixes
// make the encoding injective.  Normalisation folds ASCII A-Z to a-z,
// replaces each run of ASCII whitespace (space, \t, \n, \v, \f, \r) by one
// space and drops leading and trailing whitespace; other bytes pass through.
// The 64-bit key that feeds the dedup is the digest's first 8 bytes read
// big-endian, as a signed (two's-complement) integer.
//
// One thread per node: SHA-256 is sequential within a message, and a window
// holds thousands of nodes.  A workgroup first copies its nodes' text and
// parameter bytes into LDS; each thread then writes its message into its own
// LDS column, in rounds of three 64-byte blocks, and compresses each round's
// blocks (FIPS 180-4, Sec. 6.2).  Byte sources are read 16 bytes at a time
// through buffer descriptors, so reads past a buffer's end return zeros and
// never touch memory.
#include "common.h"

namespace hs {

typedef int i32x4s __attribute__((ext_vector_type(4)));

// FIPS 180-4 Sec. 4.2.2: first 32 bits of the fractional parts of the cube
// roots of the first 64 primes.
__device__ constexpr uint32_t kSha256K[64] = {
    0x428a2f98u, 0x71374491u, 0xb5c0fbcfu, 0xe9b5dba5u, 0x3956c25bu, 0x59f111f1u, 0x923f82a4u,
    0xab1c5ed5u, 0xd807aa98u, 0x12835b01u, 0x243185beu, 0x550c7dc3u, 0x72be5d74u, 0x80deb1feu,
    0x9bdc06a7u, 0xc19bf174u, 0xe49b69c1u, 0xefbe4786u, 0x0fc19dc6u, 0x240ca1ccu, 0x2de92c6fu,
    0x4a7484aau, 0x5cb0a9dcu, 0x76f988dau, 0x983e5152u, 0xa831c66du, 0xb00327c8u, 0xbf597fc7u,
    0xc6e00bf3u, 0xd5a79147u, 0x06ca6351u, 0x14292967u, 0x27b70a85u, 0x2e1b2138u, 0x4d2c6dfcu,
    0x53380d13u, 0x650a7354u, 0x766a0abbu, 0x81c2c92eu, 0x92722c85u, 0xa2bfe8a1u, 0xa81a664bu,
    0xc24b8b70u, 0xc76c51a3u, 0xd192e819u, 0xd6990624u, 0xf40e3585u, 0x106aa070u, 0x19a4c116u,
    0x1e376c08u, 0x2748774cu, 0x34b0bcb5u, 0x391c0cb3u, 0x4ed8aa4au, 0x5b9cca4fu, 0x682e6ff3u,
    0x748f82eeu, 0x78a5636fu, 0x84c87814u, 0x8cc70208u, 0x90befffau, 0xa4506cebu, 0xbef9a3f7u,
    0xc67178f2u};

// FIPS 180-4 Sec. 5.3.3: first 32 bits of the fractional parts of the square
// roots of the first 8 primes.
__device__ constexpr uint32_t kSha256H0[8] = {0x6a09e667u, 0xbb67ae85u, 0x3c6ef372u,
                                              0xa54ff53au, 0x510e527fu, 0x9b05688cu,
                                              0x1f83d9abu, 0x5be0cd19u};

__device__ __forceinline__ uint32_t rotr(uint32_t x, int n) {
  return (x >> n) | (x << (32 - n));
}

// One SHA-256 block: w[0..15] are the block's words (big-endian), h the state.
__device__ __forceinline__ void sha256_block(uint32_t h[8], uint32_t w[16]) {
  uint32_t a = h[0], b = h[1], c = h[2], d = h[3], e = h[4], f = h[5], g = h[6], hh = h[7];
#pragma unroll
  for (int t = 0; t < 64; ++t) {
    if (t >= 16) {   // message schedule in a rolling 16-word window
      const uint32_t w15 = w[(t - 15) & 15], w2 = w[(t - 2) & 15];
      const uint32_t s0 = rotr(w15, 7) ^ rotr(w15, 18) ^ (w15 >> 3);
      const uint32_t s1 = rotr(w2, 17) ^ rotr(w2, 19) ^ (w2 >> 10);
      w[t & 15] = w[t & 15] + s0 + w[(t - 7) & 15] + s1;
    }
    const uint32_t S1 = rotr(e, 6) ^ rotr(e, 11) ^ rotr(e, 25);
    const uint32_t ch = (e & f) ^ (~e & g);
    const uint32_t t1 = hh + S1 + ch + kSha256K[t] + w[t & 15];
    const uint32_t S0 = rotr(a, 2) ^ rotr(a, 13) ^ rotr(a, 22);
    const uint32_t mj = (a & b) ^ (a & c) ^ (b & c);
    const uint32_t t2 = S0 + mj;
    hh = g;
    g = f;
    f = e;
    e = d + t1;
    d = c;
    c = b;
    b = a;
    a = t1 + t2;
  }
  h[0] += a;
  h[1] += b;
  h[2] += c;
  h[3] += d;
  h[4] += e;
  h[5] += f;
  h[6] += g;
  h[7] += hh;
}

// 16 bytes at the 16-aligned offset `off` of a buffer of `nbytes`; bytes past
// the end read as zero.  The last partial block is read byte by byte (a
// 16-byte buffer load that straddles the end may return zeros for all of it).
__device__ __forceinline__ void load_window(__amdgpu_buffer_rsrc_t r, uint32_t off,
                                            uint32_t nbytes, uint32_t win[4]) {
  if (off + 16u <= nbytes) {
    const i32x4s v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
    win[0] = (uint32_t)v[0];
    win[1] = (uint32_t)v[1];
    win[2] = (uint32_t)v[2];
    win[3] = (uint32_t)v[3];
  } else {
    uint32_t t[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const uint32_t b =
          off + i < nbytes ? (uint32_t)__builtin_amdgcn_raw_buffer_load_b8(r, (int)(off + i), 0, 0)
                           : 0u;
      t[i >> 2] |= b << ((i & 3) * 8);
    }
    win[0] = t[0];
    win[1] = t[1];
    win[2] = t[2];
    win[3] = t[3];
  }
}

struct SigArgs {
  const uint32_t *op_type;
  const uint8_t *params;
  const int64_t *param_off;
  uint32_t param_bytes;
  const uint8_t *text;
  const int64_t *text_off;
  uint32_t text_bytes;
  const int32_t *pred_off;
  const int32_t *pred_idx;
  int64_t pred_count;
  int64_t first, count;
  int normalize;
  uint8_t *digest;
  int64_t *keys;
};

__device__ __forceinline__ void clamp_range(const int64_t *off, int64_t i, uint32_t nbytes,
                                            uint32_t &b, uint32_t &e) {
  int64_t lo = off ? off[i] : 0, hi = off ? off[i + 1] : 0;
  lo = lo < 0 ? 0 : lo > (int64_t)nbytes ? (int64_t)nbytes : lo;
  hi = hi < lo ? lo : hi > (int64_t)nbytes ? (int64_t)nbytes : hi;
  b = (uint32_t)lo;
  e = (uint32_t)hi;
}

constexpr int kSigThreads = 128;
// LDS staging of one group's text and parameter bytes
constexpr uint32_t kStageText = 16 * 1024, kStageParam = 2 * 1024;
// Messages are built in LDS in rounds of kRound bytes (three SHA-256 blocks),
// one column of kRound / 4 words per thread.
constexpr uint32_t kRound = 192;

// Stages [sb, sb + sl) of a buffer of `nbytes` (sb, sl multiples of 16) into
// LDS with coalesced 16-byte loads, eight in flight per thread; the one block
// that straddles the buffer's end is read byte by byte by thread 0.
__device__ __forceinline__ void stage_bytes(__amdgpu_buffer_rsrc_t r, uint32_t nbytes, uint32_t sb,
                                            uint32_t sl, uint4 *dst) {
  const uint32_t nch = sl >> 4;
  const uint32_t nfull = nbytes > sb ? ((nbytes - sb) >> 4 < nch ? (nbytes - sb) >> 4 : nch) : 0u;
  const int tid = threadIdx.x;
  for (uint32_t i0 = 0; i0 < nfull; i0 += kSigThreads * 8) {
    i32x4s v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const uint32_t i = i0 + u * kSigThreads + tid;
      v[u] = i < nfull ? __builtin_amdgcn_raw_buffer_load_b128(r, (int)(sb + 16u * i), 0, 0)
                       : i32x4s{0, 0, 0, 0};
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const uint32_t i = i0 + u * kSigThreads + tid;
      if (i < nfull)
        dst[i] = make_uint4((uint32_t)v[u][0], (uint32_t)v[u][1], (uint32_t)v[u][2],
                            (uint32_t)v[u][3]);
    }
  }
  if (tid == 0 && nfull < nch) {
    uint32_t w[4];
    load_window(r, sb + 16u * nfull, nbytes, w);
    dst[nfull] = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// The 16-byte window at `base` of a byte source: from the LDS copy when the
// source was staged and the window lies inside it, else from global memory.
__device__ __forceinline__ void fetch_window(bool staged, const uint4 *lds, uint32_t sb,
                                             __amdgpu_buffer_rsrc_t r, uint32_t base,
                                             uint32_t nbytes, uint32_t win[4]) {
  if (staged) {
    const uint4 x = lds[(base - sb) >> 4];
    win[0] = x.x;
    win[1] = x.y;
    win[2] = x.z;
    win[3] = x.w;
  } else {
    load_window(r, base, nbytes, win);
  }
}

template <bool NORM>
__global__ __launch_bounds__(kSigThreads) void signature_kernel(SigArgs a) {
  // all lanes read the same buffers: the descriptors are wave-uniform
  const __amdgpu_buffer_rsrc_t rp =
      __builtin_amdgcn_make_buffer_rsrc((void *)a.params, (short)0, (int)a.param_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t rt =
      __builtin_amdgcn_make_buffer_rsrc((void *)a.text, (short)0, (int)a.text_bytes, 0x00020000);
  const uint32_t dig_bytes = (uint32_t)(a.first * 32);   // digests of earlier nodes only
  const __amdgpu_buffer_rsrc_t rd =
      __builtin_amdgcn_make_buffer_rsrc((void *)a.digest, (short)0, (int)dig_bytes, 0x00020000);
  __shared__ uint4 s_text[kStageText / 16];
  __shared__ uint4 s_par[kStageParam / 16];
  __shared__ uint32_t s_msg[kRound / 4 * kSigThreads];
  const int64_t vend = a.first + a.count;

  // Groups of kSigThreads consecutive nodes.  Their texts (and parameters)
  // are consecutive in the buffers, so the group first copies the byte range
  // from its first node's start to its last node's end into LDS (the first
  // kStageText bytes of it); a thread whose text lies inside the copy reads
  // it there, any other from global memory.
  for (int64_t g0 = a.first + (int64_t)blockIdx.x * kSigThreads; g0 < vend;
       g0 += (int64_t)gridDim.x * kSigThreads) {
    const int64_t v = g0 + threadIdx.x;
    const int64_t glast = (g0 + kSigThreads < vend ? g0 + kSigThreads : vend) - 1;
    uint32_t gt0, gt1, gp0, gp1, dummy;
    clamp_range(a.text_off, g0, a.text_bytes, gt0, dummy);
    clamp_range(a.text_off, glast, a.text_bytes, dummy, gt1);
    clamp_range(a.param_off, g0, a.param_bytes, gp0, dummy);
    clamp_range(a.param_off, glast, a.param_bytes, dummy, gp1);
    const uint32_t tsb = gt0 & ~15u, psb = gp0 & ~15u;
    uint32_t tsl = gt1 > tsb ? ((gt1 - tsb + 15u) & ~15u) : 0u;
    uint32_t psl = gp1 > psb ? ((gp1 - psb + 15u) & ~15u) : 0u;
    tsl = tsl < kStageText ? tsl : kStageText;
    psl = psl < kStageParam ? psl : kStageParam;
    __syncthreads();   // the previous group is done with the copies
    stage_bytes(rt, a.text_bytes, tsb, tsl, s_text);
    stage_bytes(rp, a.param_bytes, psb, psl, s_par);
    __syncthreads();
    if (v >= vend) continue;

    const uint32_t tau = a.op_type[v];
    uint32_t p0, p1, t0, t1;
    clamp_range(a.param_off, v, a.param_bytes, p0, p1);
    clamp_range(a.text_off, v, a.text_bytes, t0, t1);
    const bool t_lds = t0 >= tsb && t1 <= tsb + tsl;
    const bool p_lds = p0 >= psb && p1 <= psb + psl;
    int64_t q0 = 0, q1 = 0;
    if (a.pred_off) {
      q0 = a.pred_off[v];
      q1 = a.pred_off[v + 1];
      q0 = q0 < 0 ? 0 : q0 > a.pred_count ? a.pred_count : q0;
      q1 = q1 < q0 ? q0 : q1 > a.pred_count ? a.pred_count : q1;
    }
    const uint32_t P = p1 - p0, m = (uint32_t)(q1 - q0);
    uint32_t win[4];
    uint32_t h[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) h[i] = kSha256H0[i];

    if (16u + P + (t1 - t0) + 32u * m + 9u <= kRound) {
      // Short message: write it into this thread's LDS column (word j at
      // s_msg[j * kSigThreads + tid], bytes in message order within a word),
      // then compress its blocks.  The column layout keeps every LDS access
      // of a wave on distinct banks.
      uint8_t *col = (uint8_t *)s_msg;
      const int tid = threadIdx.x;
      auto put8 = [&](uint32_t o, uint32_t b) {
        col[((o >> 2) * kSigThreads + tid) * 4 + (o & 3u)] = (uint8_t)b;
      };
      auto put32 = [&](uint32_t o, uint32_t x) {
#pragma unroll
        for (int i = 0; i < 4; ++i) put8(o + i, (x >> (8 * i)) & 0xffu);
      };
#pragma unroll
      for (uint32_t j = 0; j < kRound / 4; ++j) s_msg[j * kSigThreads + tid] = 0u;
      s_msg[tid] = tau;                    // le32(tau), bytes 0..3
      s_msg[kSigThreads + tid] = P;        // le32(|Theta|), bytes 4..7
      // Bytes are consumed one aligned 16-byte window at a time (every lane
      // fetches its k-th window in the same iteration), with the window's
      // bytes unrolled.  Each byte is written at the output position
      // whether or not it is kept, and the position only advances past kept
      // bytes, so a byte that is not kept is overwritten by the next one (or
      // by the field that follows).
      uint32_t o = 8u;
      uint32_t gap = 0u;
      for (uint32_t base = p0 & ~15u; base < p1; base += 16u) {
        fetch_window(p_lds, s_par, psb, rp, base, a.param_bytes, win);
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const uint32_t r = base + i;
          put8(o, (win[i >> 2] >> (8 * (i & 3))) & 0xffu);
          o += (uint32_t)(r >= p0) & (uint32_t)(r < p1);
        }
      }
      const uint32_t o0 = 12u + P;         // first byte of D
      o = o0;
      for (uint32_t base = t0 & ~15u; base < t1; base += 16u) {
        fetch_window(t_lds, s_text, tsb, rt, base, a.text_bytes, win);
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const uint32_t r = base + i;
          const uint32_t c = (win[i >> 2] >> (8 * (i & 3))) & 0xffu;
          // (bitwise & and | on the flags: no short-circuit branches)
          const uint32_t in = (uint32_t)(r >= t0) & (uint32_t)(r < t1);
          if (!NORM) {
            put8(o, c);
            o += in;
          } else {
            const uint32_t sp = (uint32_t)(c == 0x20u) | (uint32_t)(c - 0x09u < 5u);
            const uint32_t keep = in & (sp ^ 1u);
            // a kept byte after a gap is preceded by one space, unless it
            // is the first byte of D
            put8(o, 0x20u);
            o += keep & gap & (uint32_t)(o > o0);
            put8(o, c + ((uint32_t)(c - 0x41u < 26u) << 5));
            o += keep;
            gap = (in & sp) | (gap & (in ^ 1u));
          }
        }
      }
      const uint32_t D = o - o0;
      put32(8u + P, D);
      put32(o, m);
      o += 4;
      for (uint32_t j = 0; j < m; ++j) {
        const int64_t u = a.pred_idx[q0 + j];
        uint32_t d8[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
        if (u >= 0 && u < a.first) {
          load_window(rd, (uint32_t)u * 32u, dig_bytes, d8);
          load_window(rd, (uint32_t)u * 32u + 16u, dig_bytes, d8 + 4);
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) put32(o + 4 * i, d8[i]);
        o += 32;
      }
      const uint32_t L = o;
      const uint32_t nblk = (L + 8u) / 64u + 1u;
      put8(L, 0x80u);
      const uint64_t bits = (uint64_t)L * 8u;
      // last 8 bytes: bit length, big-endian (the high three are zero)
      const uint32_t e8 = nblk * 64u - 8u;
#pragma unroll
      for (int i = 3; i < 8; ++i) put8(e8 + i, (uint32_t)(bits >> (8 * (7 - i))) & 0xffu);
      for (uint32_t bk = 0; bk < nblk; ++bk) {
        uint32_t w[16];
#pragma unroll
        for (int i = 0; i < 16; ++i)
          w[i] = __builtin_bswap32(s_msg[(bk * 16u + i) * kSigThreads + tid]);
        sha256_block(h, w);
      }
    } else {
      // Longer message: the same column, filled and compressed in rounds.
      // The message is built in this thread's LDS column in rounds of
      // kRound bytes (word j of a round at s_msg[j * kSigThreads + tid], bytes
      // in message order within a word; the column layout keeps every LDS
      // access of a wave on distinct banks), and each round's blocks are then
      // compressed.  Every writer places bytes by their message position and
      // a round keeps those inside it.  Source bytes are consumed one aligned
      // 16-byte window at a time (every lane takes its k-th window in the same
      // iteration), with the window's bytes unrolled.
      uint8_t *col = (uint8_t *)s_msg;
      const int tid = threadIdx.x;
      uint32_t r0 = 0, r_end = 0;
      auto put8 = [&](uint32_t o, uint32_t b) {
        if (o >= r0 && o < r_end)
          col[(((o - r0) >> 2) * kSigThreads + tid) * 4 + (o & 3u)] = (uint8_t)b;
      };
      auto put32 = [&](uint32_t o, uint32_t x) {
  #pragma unroll
        for (int i = 0; i < 4; ++i) put8(o + i, (x >> (8 * i)) & 0xffu);
      };

      // |D| comes before D in the message: with normalisation, count it first
      uint32_t D = t1 - t0;
      if (NORM) {
        D = 0;
        uint32_t gap = 0;
        for (uint32_t base = t0 & ~15u; base < t1; base += 16u) {
          fetch_window(t_lds, s_text, tsb, rt, base, a.text_bytes, win);
  #pragma unroll
          for (int i = 0; i < 16; ++i) {
            const uint32_t r = base + i;
            const uint32_t c = (win[i >> 2] >> (8 * (i & 3))) & 0xffu;
            const uint32_t in = (uint32_t)(r >= t0) & (uint32_t)(r < t1);
            const uint32_t sp = (uint32_t)(c == 0x20u) | (uint32_t)(c - 0x09u < 5u);
            const uint32_t keep = in & (sp ^ 1u);
            D += keep & gap & (uint32_t)(D > 0u);
            D += keep;
            gap = (in & sp) | (gap & (in ^ 1u));
          }
        }
      }
      const uint32_t o0 = 12u + P;                  // first byte of D
      const uint32_t L = 16u + P + D + 32u * m;     // message bytes
      const uint32_t end = ((L + 8u) / 64u + 1u) * 64u;
      const uint64_t bits = (uint64_t)L * 8u;
      // resume point of the normalised text: start of the last window taken
      uint32_t n_base = t0 & ~15u, n_o = o0, n_gap = 0;

      for (r0 = 0; r0 < end; r0 += kRound) {
        r_end = r0 + kRound < end ? r0 + kRound : end;
  #pragma unroll
        for (uint32_t j = 0; j < kRound / 4; ++j) s_msg[j * kSigThreads + tid] = 0u;
        put32(0u, tau);
        put32(4u, P);
        // parameters: message bytes 8 .. 8 + P (only the windows this round needs)
        if (8u + P > r0 && 8u < r_end) {
          const uint32_t i0 = r0 > 8u ? r0 - 8u : 0u;
          const uint32_t i1 = r_end - 8u < P ? r_end - 8u : P;
          for (uint32_t base = (p0 + i0) & ~15u; base < p0 + i1; base += 16u) {
            fetch_window(p_lds, s_par, psb, rp, base, a.param_bytes, win);
  #pragma unroll
            for (int i = 0; i < 16; ++i) {
              const uint32_t r = base + i;
              if (r >= p0 && r < p1) put8(8u + r - p0, (win[i >> 2] >> (8 * (i & 3))) & 0xffu);
            }
          }
        }
        if (!NORM) {
          if (o0 + D > r0 && o0 < r_end) {
            const uint32_t i0 = r0 > o0 ? r0 - o0 : 0u;
            const uint32_t i1 = r_end - o0 < D ? r_end - o0 : D;
            for (uint32_t base = (t0 + i0) & ~15u; base < t0 + i1; base += 16u) {
              fetch_window(t_lds, s_text, tsb, rt, base, a.text_bytes, win);
  #pragma unroll
              for (int i = 0; i < 16; ++i) {
                const uint32_t r = base + i;
                if (r >= t0 && r < t1) put8(o0 + r - t0, (win[i >> 2] >> (8 * (i & 3))) & 0xffu);
              }
            }
          }
        } else {
          // Each byte is written at the output position whether or not it is
          // kept; the position only advances past kept bytes, so a byte that
          // is not kept is overwritten by the next one (or by the field that
          // follows D).  A window that runs past the round is taken again,
          // from the state saved at its start, by the next round.
          uint32_t base = n_base, o = n_o, gap = n_gap;
          while (base < t1 && o < r_end) {
            n_base = base;
            n_o = o;
            n_gap = gap;
            fetch_window(t_lds, s_text, tsb, rt, base, a.text_bytes, win);
  #pragma unroll
            for (int i = 0; i < 16; ++i) {
              const uint32_t r = base + i;
              const uint32_t c = (win[i >> 2] >> (8 * (i & 3))) & 0xffu;
              // (bitwise & and | on the flags: no short-circuit branches)
              const uint32_t in = (uint32_t)(r >= t0) & (uint32_t)(r < t1);
              const uint32_t sp = (uint32_t)(c == 0x20u) | (uint32_t)(c - 0x09u < 5u);
              const uint32_t keep = in & (sp ^ 1u);
              // a kept byte after a gap is preceded by one space, unless it is
              // the first byte of D
              put8(o, 0x20u);
              o += keep & gap & (uint32_t)(o > o0);
              put8(o, c + ((uint32_t)(c - 0x41u < 26u) << 5));
              o += keep;
              gap = (in & sp) | (gap & (in ^ 1u));
            }
            base += 16u;
          }
        }
        put32(8u + P, D);
        put32(o0 + D, m);
        // predecessor digests: message bytes 16 + P + D + 32 j
        for (uint32_t j = 0; j < m; ++j) {
          const uint32_t oj = 16u + P + D + 32u * j;
          if (oj + 32u <= r0 || oj >= r_end) continue;
          const int64_t u = a.pred_idx[q0 + j];
          uint32_t d8[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
          if (u >= 0 && u < a.first) {
            load_window(rd, (uint32_t)u * 32u, dig_bytes, d8);
            load_window(rd, (uint32_t)u * 32u + 16u, dig_bytes, d8 + 4);
          }
  #pragma unroll
          for (int i = 0; i < 8; ++i) put32(oj + 4 * i, d8[i]);
        }
        put8(L, 0x80u);
        // last 8 bytes: the bit length, big-endian (the high three are zero)
  #pragma unroll
        for (int i = 3; i < 8; ++i) put8(end - 8u + i, (uint32_t)(bits >> (8 * (7 - i))) & 0xffu);
        for (uint32_t bk = 0; bk < (r_end - r0) / 64u; ++bk) {
          uint32_t w[16];
  #pragma unroll
          for (int i = 0; i < 16; ++i)
            w[i] = __builtin_bswap32(s_msg[(bk * 16u + i) * kSigThreads + tid]);
          sha256_block(h, w);
        }
      }
    }

    uint4 *dst = (uint4 *)(a.digest + v * 32);
    dst[0] = make_uint4(__builtin_bswap32(h[0]), __builtin_bswap32(h[1]),
                        __builtin_bswap32(h[2]), __builtin_bswap32(h[3]));
    dst[1] = make_uint4(__builtin_bswap32(h[4]), __builtin_bswap32(h[5]),
                        __builtin_bswap32(h[6]), __builtin_bswap32(h[7]));
    if (a.keys) a.keys[v] = (int64_t)(((uint64_t)h[0] << 32) | h[1]);
  }
}

hipError_t launch_signature(const uint32_t *op_type, const uint8_t *params,
                            const int64_t *param_off, int64_t param_bytes, const uint8_t *text,
                            const int64_t *text_off, int64_t text_bytes, const int32_t *pred_off,
                            const int32_t *pred_idx, int64_t pred_count, int64_t first,
                            int64_t count, int normalize, uint8_t *digest, int64_t *keys,
                            hipStream_t st) {
  if (count <= 0) return hipSuccess;
  SigArgs a;
  a.op_type = op_type;
  a.params = params;
  a.param_off = param_off;
  a.param_bytes = (uint32_t)param_bytes;
  a.text = text;
  a.text_off = text_off;
  a.text_bytes = (uint32_t)text_bytes;
  a.pred_off = pred_off;
  a.pred_idx = pred_idx;
  a.pred_count = pred_count;
  a.first = first;
  a.count = count;
  a.normalize = normalize;
  a.digest = digest;
  a.keys = keys;
  int64_t blocks = (count + kSigThreads - 1) / kSigThreads;
  if (blocks > 8192) blocks = 8192;
  if (normalize)
    hipLaunchKernelGGL(signature_kernel<true>, dim3((unsigned)blocks), dim3(kSigThreads), 0, st, a);
  else
    hipLaunchKernelGGL(signature_kernel<false>, dim3((unsigned)blocks), dim3(kSigThreads), 0, st,
                       a);
  return hipGetLastError();
}

}  // namespace hs
