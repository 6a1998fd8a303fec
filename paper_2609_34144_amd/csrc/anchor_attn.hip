// Routed block-sparse anchor attention on gfx950 (Sec. 4.4; App. B.4).
//
// Flash-style single pass with bf16 MFMA (v_mfma_f32_32x32x16_bf16) and fp32
// online softmax.  One workgroup = 4 waves = 128 queries of one (anchor, head);
// each wave owns 32 queries.  The key sequence of the (anchor, head) is the
// concatenation [current segment (n0 tokens) ; routed chunk idx[0] ; ... ], walked
// in tiles of 64 keys.
//
// Data movement: every K and V tile is copied global -> LDS by the buffer unit
// (buffer_load_dwordx4 ... lds), so no registers or VALU work stage it.  Each
// lane of a copy instruction picks its source row and 16-byte chunk, which lets
// the LDS image be XOR-swizzled against bank conflicts even though the copy
// writes 1 KB contiguously.  Two K and two V buffers rotate; one barrier per tile.
//
// Per wave and tile:
//   S^T = K Q^T   A = K rows from LDS (ds_read_b128), B = Q^T held in registers
//                 for the whole kernel.  The 32x32 accumulator puts one query per
//                 lane column, so the online-softmax row max / row sum need only
//                 the lane's own values and one exchange with lane ^ 32.
//   O^T += V^T P^T  B = P^T straight from the S^T accumulators (converted to
//                 bf16; the contraction index order is free, so no data moves),
//                 A = V^T read from the row-major V tile with the transposing
//                 LDS load ds_read_b64_tr_b16.
// Software pipeline: iteration j issues the copies of K[j+2] and V[j], the
// MFMAs of S[j+1] = K[j+1] Q^T and of O += P[j-1] V[j-1], and the softmax of S[j]
// (VALU); the three are independent, so the matrix cores and the VALU overlap
// inside one wave.
// Blocks are renumbered so that the Q-tiles of one (anchor, head) land on the
// same XCD and share its L2 for the routed K/V.
#include "cast_common.h"

namespace cast {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
typedef __attribute__((address_space(3))) char lds_char;

constexpr int kBK = 64;    // keys per tile
constexpr int kThreads = 256;
constexpr int kMaxKeff = kAttnMaxKeff;   // routed chunk indices cached in LDS
// The running max used for the exponentials moves only when the tile max exceeds
// it by more than this (log2 units): probabilities stay <= 2^8, harmless in fp32
// sums and bf16 operands, and the O rescale is skipped for most tiles.
constexpr float kMaxSlack = 8.0f;

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* idx;
  const uint16_t* kc;
  const uint16_t* vc;
  uint16_t* out;
  float* lse;
  int n_a, S, H, M, Bv, n0, k_eff, L, n_qt, nblocks;
  unsigned long long bv_magic;   // ceil(2^40 / Bv): row / Bv = (row * magic) >> 40
  float sl2;                     // scale * log2(e)
  long long hist_bytes;          // extent of the K/V history tensors
  long long cur_bytes;           // extent of the current-segment K/V tensors
};

template <int V>
struct IC {
  static constexpr int value = V;
};

template <int B, int E, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(IC<B>{});
    static_for<B + 1, E>(f);
  }
}

// Block b runs on XCD b % 8; give each XCD a contiguous range of logical blocks.
__device__ __forceinline__ int xcd_remap(int b, int nb) {
  const int per = nb / 8, rem = nb % 8;
  const int xcd = b % 8, j = b / 8;
  return (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + j;
}

// Two floats -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

constexpr int kBufDword3 = 0x00020000;   // 32-bit data format, gfx9-family V#

__device__ __forceinline__ __amdgpu_buffer_rsrc_t tensor_rsrc(const void* base, long long bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0,
                                           (int)(unsigned)(bytes < 0xffffffffll ? bytes : 0xffffffffll),
                                           kBufDword3);
}

template <int DH>
struct Geo {
  static constexpr int CPR = DH / 8;                     // 16-byte chunks per row
  static constexpr int ROWB = DH * 2;                    // bytes per row
  static constexpr int TILEB = kBK * ROWB;               // bytes per K or V tile
  static constexpr int DPT = TILEB / (kThreads * 16);    // copy instructions per thread per tile
};

// LDS swizzles (chunk c of tile row r is stored at chunk c ^ swz(r)):
//  K: a ds_read_b128 of one logical chunk by 32 consecutive rows; XOR by r mod CPR
//     spreads any 16 consecutive rows over 16 distinct 16-byte bank groups.
//  V: a transposing read takes 4 consecutive rows x 32 bytes per 16 lanes, the
//     two 16-lane halves of 32 lanes 32 bytes apart; XOR by {0, 10, 4, 14}[r mod 4]
//     gives the 8 row segments of 32 lanes 8 distinct 32-byte bank groups.
__device__ __forceinline__ constexpr int kswz(int r, int cpr) { return r & (cpr - 1); }
__device__ __forceinline__ constexpr int vswz(int r, int cpr) {
  return ((2 * (r & 3)) ^ (8 * (r & 1))) & (cpr - 1);
}

// FAST: no current segment and chunks of >= 64 rows, so every tile takes the
// uniform two-chunk mapping and its copies can be issued inside the MFMA block.
template <int DH, bool FAST>
__global__ __launch_bounds__(kThreads, 2) void anchor_attn_kernel(AttnArgs a) {
  using G = Geo<DH>;
  // separate objects, so the compiler can tell the copy targets from the buffers
  // being read and does not wait for in-flight copies before unrelated LDS reads
  __shared__ __attribute__((aligned(1024))) uint16_t lds_k0[kBK * DH];
  __shared__ __attribute__((aligned(1024))) uint16_t lds_k1[kBK * DH];
  __shared__ __attribute__((aligned(1024))) uint16_t lds_v0[kBK * DH];
  __shared__ __attribute__((aligned(1024))) uint16_t lds_v1[kBK * DH];
  __shared__ int sidx[kMaxKeff + 1];

  const int logical = xcd_remap(blockIdx.x, a.nblocks);
  const int pair = logical / a.n_qt, qt = logical - pair * a.n_qt;
  const int i = pair / a.H, h = pair - (pair / a.H) * a.H;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hf = lane >> 5;
  // routed chunk indices of this (anchor, head), clamped into [0, M)
  // (entry k_eff repeats the last one, so a tile's "next slot" always names a real chunk)
  if (a.k_eff > 0) {
    const int32_t* idx_ih = a.idx + ((long long)i * a.H + h) * a.k_eff;
    for (int j = tid; j <= a.k_eff; j += kThreads) {
      const int c = idx_ih[j < a.k_eff ? j : a.k_eff - 1];
      sidx[j] = c < 0 ? 0 : (c >= a.M ? a.M - 1 : c);
    }
  } else if (tid < 2) {
    sidx[tid] = 0;
  }

  // ---- Q^T operand in registers: the lane holds query qt*128 + wave*32 + l32,
  //      d = 16t + 8hf .. +8
  bf16x8 qreg[DH / 16];
  {
    const int qi = qt * 128 + wave * 32 + l32;
    // rows past S load the last query; their outputs are never stored
    const int qc = qi < a.S ? qi : a.S - 1;
    const uint16_t* qp = a.q + (((long long)i * a.S + qc) * a.H + h) * DH + 8 * hf;
#pragma unroll
    for (int t = 0; t < DH / 16; ++t)
      qreg[t] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(qp + 16 * t));
  }
  __syncthreads();   // sidx visible to every wave

  const unsigned row_bytes = (unsigned)(a.H * DH * 2), head_bytes = (unsigned)(h * DH * 2);

  // ---- copy slots: instruction n of this wave fills LDS chunk
  //      ci = (wave * DPT + n) * 64 + lane of a tile, i.e. row ci / CPR and
  //      physical chunk ci % CPR, which holds logical chunk (ci % CPR) ^ swz(row)
  auto slot_row = [&](int n) __attribute__((always_inline)) -> int {
    return ((wave * G::DPT + n) * 64 + lane) / G::CPR;
  };
  auto slot_off = [&](int n, bool is_v) __attribute__((always_inline)) -> unsigned {
    const int r = slot_row(n), pc = lane % G::CPR;
    return (unsigned)((pc ^ (is_v ? vswz(r, G::CPR) : kswz(r, G::CPR))) * 16);
  };
  auto copy16 = [&](__amdgpu_buffer_rsrc_t rs, uint16_t* dst, int n, unsigned off)
      __attribute__((always_inline)) {
    // recomputed at each use (the laundering stops the compiler from keeping the
    // 16 LDS bases of all buffers live in scalar registers across the loop)
    int wbase = wave * G::DPT * 1024;
    asm volatile("" : "+s"(wbase));
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rs, (lds_void*)(reinterpret_cast<char*>(dst) + wbase + n * 1024), 16, (int)off, 0, 0, 0);
  };
  // Copy tile `tile` of K (IsV = 0) or V (IsV = 1) into `dst`.  Row j of the tile is
  // sequence row r = 64*tile + j: current segment rows r < n0, then routed chunk
  // rows.  History-only tiles with chunks of >= 64 rows meet at most two routed
  // slots s0, s0 + 1, whose rows are contiguous, so row j sits at
  // (j < split ? base0 : base1) + j * row_bytes with wave-uniform base0, base1,
  // split.  Rows past the end read real rows (clamped, or of the padded slot);
  // their logits are masked to -inf and add nothing.
  struct TileMap { unsigned base0, base1; int split; };
  auto tile_map = [&](int tile) __attribute__((always_inline)) -> TileMap {
    const int u0 = tile * kBK - a.n0;                     // first chunk-part row of the tile
    const int s0 = u0 / a.Bv, tb = s0 * a.Bv;
    const int c0 = __builtin_amdgcn_readfirstlane(sidx[s0]);
    const int c1 = __builtin_amdgcn_readfirstlane(sidx[s0 + 1]);
    TileMap m;
    m.base0 = (unsigned)(c0 * a.Bv + (u0 - tb)) * row_bytes + head_bytes;
    m.base1 = (unsigned)(c1 * a.Bv + (u0 - tb - a.Bv)) * row_bytes + head_bytes;
    m.split = tb + a.Bv - u0;
    return m;
  };
  auto copy_fast = [&](auto is_v, const TileMap& m, int n, uint16_t* dst) __attribute__((always_inline)) {
    constexpr bool IsV = decltype(is_v)::value != 0;
    const int r = slot_row(n);
    const unsigned off = (r < m.split ? m.base0 : m.base1) + (unsigned)r * row_bytes + slot_off(n, IsV);
    copy16(tensor_rsrc(IsV ? a.v : a.k, a.hist_bytes), dst, n, off);
  };
  auto load_tile = [&](auto is_v, int tile, uint16_t* dst) __attribute__((always_inline)) {
    constexpr bool IsV = decltype(is_v)::value != 0;
    const __amdgpu_buffer_rsrc_t rh = tensor_rsrc(IsV ? a.v : a.k, a.hist_bytes);
    if (FAST || (tile * kBK >= a.n0 && a.Bv >= kBK)) {
      const TileMap m = tile_map(tile);
#pragma unroll
      for (int n = 0; n < G::DPT; ++n) copy_fast(is_v, m, n, dst);
    } else {
      // tiles that touch the current segment, or chunks shorter than a tile:
      // per-row slot by multiply-shift
#pragma unroll
      for (int n = 0; n < G::DPT; ++n) {
        int r = tile * kBK + slot_row(n);
        r = r < a.L ? r : a.L - 1;
        const unsigned co = slot_off(n, IsV);
        const int rr = max(r - a.n0, 0);
        const int slot = (int)(((unsigned long long)(unsigned)rr * a.bv_magic) >> 40);
        const int t = rr - slot * a.Bv;
        const unsigned hoff = (unsigned)(sidx[slot] * a.Bv + t) * row_bytes + head_bytes + co;
        // two copies under complementary lane masks (not an if/else, which would be
        // merged into one copy with a per-lane descriptor)
        if (r < a.n0)
          copy16(tensor_rsrc(IsV ? a.vc : a.kc, a.cur_bytes), dst, n,
                 (unsigned)r * row_bytes + head_bytes + co);
        if (r >= a.n0) copy16(rh, dst, n, hoff);
      }
    }
  };

  // ---- LDS read addresses (bytes within a tile)
  // K: lane reads row kb*32 + l32, logical chunk 2t + hf, stored at chunk
  // (2t + hf) ^ (l32 % CPR); as bytes that is kbase ^ 32t (the row offset is a
  // multiple of the row length, so the XOR only touches the chunk bits)
  const unsigned kbase = (unsigned)(l32 * G::ROWB + ((hf ^ kswz(l32, G::CPR)) * 16));
  // V (transposing read): within each 16-lane group gq = lane / 16, lane a supplies
  // row 4*(gq/2) + a/4 (+ 32kb + 16s + 8run) and columns d = 32db + 16(gq%2) + 4(a%4)
  // .. +4; the read returns to lane a the 4 rows' values at d = 32db + 16(gq%2) + a,
  // i.e. to every lane the column d = 32db + l32 for 4 consecutive keys.
  // As bytes: vbase ^ 64db (the row swizzle of vr only touches the chunk bits).
  unsigned vbase;
  {
    const int gq = lane >> 4, la = lane & 15;
    const int vr = 4 * (gq >> 1) + (la >> 2);
    const int c = 2 * (gq & 1) + ((la & 3) >> 1);
    vbase = (unsigned)(vr * G::ROWB + ((c ^ vswz(vr, G::CPR)) * 16) + 8 * (la & 1));
  }

  f32x16 acc_o[DH / 32];
#pragma unroll
  for (int db = 0; db < DH / 32; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc_o[db][e] = 0.0f;
  float m_run = -INFINITY, l_run = 0.0f;

  // S^T = K Q^T for the 64 keys of the tile in `kt`
  auto qk = [&](const uint16_t* kt, f32x16 (&acc)[2]) __attribute__((always_inline)) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[kb][e] = 0.0f;
    const char* kb0 = reinterpret_cast<const char*>(kt);
#pragma unroll
    for (int t = 0; t < DH / 16; ++t)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const bf16x8 ka = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(kb0 + (kbase ^ (32u * t)) + kb * 32 * G::ROWB));
        acc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qreg[t], acc[kb], 0, 0, 0);
      }
  };
  // O^T += V^T P^T for the tile in `vt`.  MFMA (kb, s) contracts the keys
  // 32kb + 16s + 4hf + {0..3} and 32kb + 16s + 8 + 4hf + {0..3}: the S^T accumulator
  // rows that lane holds as p[8s .. 8s+7] of block kb.
  auto pv = [&](const uint16_t* vt, const bf16x8 (&pb)[2][2]) __attribute__((always_inline)) {
    const lds_char* vb0 = (const lds_char*)(vt);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int db = 0; db < DH / 32; ++db) {
          const lds_char* p = vb0 + (vbase ^ (64u * db)) + (32 * kb + 16 * s) * G::ROWB;
          const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)p);
          const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p + 8 * G::ROWB));
          const bf16x8 va = __builtin_bit_cast(
              bf16x8, u32x4{__builtin_bit_cast(u32x2, lo).x, __builtin_bit_cast(u32x2, lo).y,
                            __builtin_bit_cast(u32x2, hi).x, __builtin_bit_cast(u32x2, hi).y});
          acc_o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[kb][s], acc_o[db], 0, 0, 0);
        }
  };
  // online softmax of tile `tile` (log2 domain), one query per lane column
  auto softmax = [&](f32x16 (&acc)[2], int tile, bf16x8 (&pb)[2][2], float& corr, bool& grew,
                     auto mask) __attribute__((always_inline)) {
    const int key0 = tile * kBK;
    if (decltype(mask)::value) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = key0 + kb * 32 + 8 * (e / 4) + 4 * hf + (e % 4);
          if (key >= a.L) acc[kb][e] = -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, acc[kb][e]);
    {
      const u32x2 sw = __builtin_bit_cast(
          u32x2, __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, mx),
                                                  __builtin_bit_cast(unsigned, mx), false, false));
      mx = fmaxf(__builtin_bit_cast(float, sw.x), __builtin_bit_cast(float, sw.y));
    }
    const float m_cand = fmaxf(m_run, mx * a.sl2);
    const bool up = m_cand > m_run + kMaxSlack;
    const float m_new = up ? m_cand : m_run;
    grew = __ballot(up) != 0ull;
    corr = __builtin_amdgcn_exp2f(m_run - m_new);
    float rs = 0.0f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      float p[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        p[e] = __builtin_amdgcn_exp2f(fmaf(acc[kb][e], a.sl2, -m_new));
        rs += p[e];
      }
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const u32x4 w = u32x4{pack_bf16x2(p[8 * s + 0], p[8 * s + 1]), pack_bf16x2(p[8 * s + 2], p[8 * s + 3]),
                              pack_bf16x2(p[8 * s + 4], p[8 * s + 5]), pack_bf16x2(p[8 * s + 6], p[8 * s + 7])};
        pb[kb][s] = __builtin_bit_cast(bf16x8, w);
      }
    }
    l_run = l_run * corr + rs;
    m_run = m_new;
  };

  const int nt = (a.L + kBK - 1) / kBK;
  f32x16 s0[2], s1[2];          // S^T of even / odd tiles
  bf16x8 p0[2][2], p1[2][2];    // P^T of even / odd tiles
  float c0 = 1.0f, c1 = 1.0f;   // their O rescale factors
  bool g0 = false, g1 = false;  // ... and whether any lane's max moved

  // Iteration j: copies of K[j+2] -> K buffer j%2 and V[j] -> V buffer j%2 (both
  // free: their last readers ran in iteration j-1), S[j+1] from K buffer (j+1)%2,
  // O += P[j-1] V[j-1] from V buffer (j-1)%2, softmax of S[j].  The flags say
  // which of the three are present (first, steady, last, drain iterations); in
  // the steady state the MFMA and softmax work is one straight-line block.
  enum { kQK = 1, kPV = 2, kSM = 4, kMask = 8 };
  // Steady-state block, software-ordered: MFMA u (S MFMAs, then PV MFMAs) is
  // followed by the LDS operand read of MFMA u + kLA and by slice u of the
  // softmax of the previous tile, and a scheduling barrier closes each slice, so
  // the VALU work issues while the matrix core runs and only kLA + 1 operands are
  // in flight.  Softmax slices: 0-3 partial row maxima, 4 the exchange with the
  // other half-wave and the new running max, 5-20 two exponentials each (packed to
  // bf16 every 8), 21 the running sum.
  auto fused = [&](const uint16_t* kt, f32x16 (&sn)[2], const uint16_t* vt,
                   const bf16x8 (&pp)[2][2], f32x16 (&sc)[2], bf16x8 (&pc)[2][2], float& cc,
                   bool& gc, uint16_t* kdst, int tk, uint16_t* vdst, int tv)
      __attribute__((always_inline)) {
    constexpr int NQ = 2 * (DH / 16), ND = DH / 32, NP = 4 * ND, NM = NQ + NP;
    constexpr int NS = 22, NU = NM > NS ? NM : NS, kLA = 3;
    TileMap mk{}, mv{};
    if constexpr (FAST) {
      mk = tile_map(tk);
      mv = tile_map(tv);
    }
    const char* kb0 = reinterpret_cast<const char*>(kt);
    const lds_char* vb0 = (const lds_char*)(vt);
    bf16x8 op[NM];
    float pm[4], m_new = 0.0f, rs = 0.0f;
    float pe[32];
    auto read = [&](auto uu) __attribute__((always_inline)) {
      constexpr int u = decltype(uu)::value;
      if constexpr (u < NQ) {
        constexpr int t = u / 2, kb = u % 2;
        op[u] = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(kb0 + (kbase ^ (32u * t)) + kb * 32 * G::ROWB));
      } else {
        constexpr int w = u - NQ, kb = w / (2 * ND), s2 = (w / ND) % 2, db = w % ND;
        const lds_char* p = vb0 + (vbase ^ (64u * db)) + (32 * kb + 16 * s2) * G::ROWB;
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)p);
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p + 8 * G::ROWB));
        op[u] = __builtin_bit_cast(
            bf16x8, u32x4{__builtin_bit_cast(u32x2, lo).x, __builtin_bit_cast(u32x2, lo).y,
                          __builtin_bit_cast(u32x2, hi).x, __builtin_bit_cast(u32x2, hi).y});
      }
    };
    auto mma = [&](auto uu) __attribute__((always_inline)) {
      constexpr int u = decltype(uu)::value;
      if constexpr (u < NQ) {
        constexpr int t = u / 2, kb = u % 2;
        sn[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            op[u], qreg[t], t == 0 ? f32x16{} : sn[kb], 0, 0, 0);
      } else {
        constexpr int w = u - NQ, kb = w / (2 * ND), s2 = (w / ND) % 2, db = w % ND;
        acc_o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(op[u], pp[kb][s2], acc_o[db], 0, 0, 0);
      }
    };
    auto smx = [&](auto cc_) __attribute__((always_inline)) {
      constexpr int c = decltype(cc_)::value;
      if constexpr (c < 4) {
        float m = sc[c / 2][8 * (c % 2)];
#pragma unroll
        for (int e = 1; e < 8; ++e) m = fmaxf(m, sc[c / 2][8 * (c % 2) + e]);
        pm[c] = m;
      } else if constexpr (c == 4) {
        float mx = fmaxf(fmaxf(pm[0], pm[1]), fmaxf(pm[2], pm[3]));
        const u32x2 sw = __builtin_bit_cast(
            u32x2, __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, mx),
                                                    __builtin_bit_cast(unsigned, mx), false, false));
        mx = fmaxf(__builtin_bit_cast(float, sw.x), __builtin_bit_cast(float, sw.y));
        const float m_cand = fmaxf(m_run, mx * a.sl2);
        const bool up = m_cand > m_run + kMaxSlack;
        m_new = up ? m_cand : m_run;
        gc = __ballot(up) != 0ull;
        cc = __builtin_amdgcn_exp2f(m_run - m_new);
      } else if constexpr (c < 21) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          constexpr int e = 2 * (c - 5);
          pe[e + q] = __builtin_amdgcn_exp2f(fmaf(sc[(e + q) / 16][(e + q) % 16], a.sl2, -m_new));
          rs += pe[e + q];
        }
        if constexpr ((2 * (c - 5) + 2) % 8 == 0) {
          constexpr int g = (2 * (c - 5)) / 8, o = 8 * g;
          pc[g / 2][g % 2] = __builtin_bit_cast(
              bf16x8, u32x4{pack_bf16x2(pe[o + 0], pe[o + 1]), pack_bf16x2(pe[o + 2], pe[o + 3]),
                            pack_bf16x2(pe[o + 4], pe[o + 5]), pack_bf16x2(pe[o + 6], pe[o + 7])});
          // pinned here: the values are read only in the next iteration, and the
          // compiler would otherwise sink this work out of the block it overlaps
          asm volatile("" ::"v"(pc[g / 2][g % 2]));
        }
      } else {
        l_run = l_run * cc + rs;
        m_run = m_new;
        asm volatile("" ::"v"(l_run), "v"(cc));
      }
    };
    static_for<0, kLA>([&](auto u) { read(u); });
    static_for<0, NU>([&](auto uu) {
      constexpr int u = decltype(uu)::value;
      if constexpr (FAST && u < G::DPT) copy_fast(IC<0>{}, mk, u, kdst);
      if constexpr (FAST && u >= G::DPT && u < 2 * G::DPT) copy_fast(IC<1>{}, mv, u - G::DPT, vdst);
      if constexpr (u + kLA < NM) read(IC<u + kLA>{});
      if constexpr (u < NM) mma(uu);
      if constexpr (u < NS) smx(uu);
      __builtin_amdgcn_sched_barrier(0);
    });
  };
  auto step = [&](auto par, auto flags, int j, f32x16 (&sc)[2], f32x16 (&sn)[2],
                  bf16x8 (&pp)[2][2], bf16x8 (&pc)[2][2], float& cp, bool& gp, float& cc, bool& gc)
      __attribute__((always_inline)) {
    constexpr int B = decltype(par)::value, F = decltype(flags)::value;
    uint16_t* const kmine = B == 0 ? lds_k0 : lds_k1;
    const uint16_t* const kother = B == 0 ? lds_k1 : lds_k0;
    uint16_t* const vmine = B == 0 ? lds_v0 : lds_v1;
    const uint16_t* const vother = B == 0 ? lds_v1 : lds_v0;
    __builtin_amdgcn_s_waitcnt(0);   // this wave's copies of the previous iteration landed
    __syncthreads();                 // ... and everyone's; previous readers are done
    constexpr bool kSteady = F == (kQK | kPV | kSM);
    if constexpr (!(FAST && kSteady)) {
      if ((F & kQK) && j + 2 < nt) load_tile(IC<0>{}, j + 2, kmine);
      if (F & kSM) load_tile(IC<1>{}, j, vmine);
    }
    if ((F & kPV) && gp) {
#pragma unroll
      for (int db = 0; db < DH / 32; ++db)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc_o[db][e] *= cp;
    }
    if constexpr (kSteady) {
      // (FAST: a copy of K past the end re-copies the last tile into a buffer
      // that is not read again)
      fused(kother, sn, vother, pp, sc, pc, cc, gc, kmine, min(j + 2, nt - 1), vmine, j);
    } else {
      if (F & kQK) qk(kother, sn);
      if (F & kPV) pv(vother, pp);
      if (F & kSM) softmax(sc, j, pc, cc, gc, IC<(F & kMask) ? 1 : 0>{});
    }
  };

  load_tile(IC<0>{}, 0, lds_k0);
  if (nt > 1) load_tile(IC<0>{}, 1, lds_k1);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  qk(lds_k0, s0);
  if (nt == 1) {
    step(IC<0>{}, IC<kSM | kMask>{}, 0, s0, s1, p1, p0, c1, g1, c0, g0);
    step(IC<1>{}, IC<kPV>{}, 1, s1, s0, p0, p1, c0, g0, c1, g1);
  } else {
    step(IC<0>{}, IC<kQK | kSM>{}, 0, s0, s1, p1, p0, c1, g1, c0, g0);
    int j = 1;
    for (; j + 1 <= nt - 2; j += 2) {
      step(IC<1>{}, IC<kQK | kPV | kSM>{}, j, s1, s0, p0, p1, c0, g0, c1, g1);
      step(IC<0>{}, IC<kQK | kPV | kSM>{}, j + 1, s0, s1, p1, p0, c1, g1, c0, g0);
    }
    if (j <= nt - 2) {
      step(IC<1>{}, IC<kQK | kPV | kSM>{}, j, s1, s0, p0, p1, c0, g0, c1, g1);
      ++j;
    }
    // j == nt - 1: last softmax (masked), then the drain iteration nt
    if (j & 1) {
      step(IC<1>{}, IC<kPV | kSM | kMask>{}, j, s1, s0, p0, p1, c0, g0, c1, g1);
      step(IC<0>{}, IC<kPV>{}, j + 1, s0, s1, p1, p0, c1, g1, c0, g0);
    } else {
      step(IC<0>{}, IC<kPV | kSM | kMask>{}, j, s0, s1, p1, p0, c1, g1, c0, g0);
      step(IC<1>{}, IC<kPV>{}, j + 1, s1, s0, p0, p1, c0, g0, c1, g1);
    }
  }

  // ---- epilogue: normalise, write O (bf16) and the log-sum-exp
  {
    const int qi = qt * 128 + wave * 32 + l32;
    const float l_tot = l_run + __shfl_xor(l_run, 32);
    const float inv = 1.0f / l_tot;
    if (qi < a.S) {
      uint16_t* op = a.out + (((long long)i * a.S + qi) * a.H + h) * DH + 4 * hf;
#pragma unroll
      for (int db = 0; db < DH / 32; ++db)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const u32x2 w = u32x2{pack_bf16x2(acc_o[db][4 * g4 + 0] * inv, acc_o[db][4 * g4 + 1] * inv),
                                pack_bf16x2(acc_o[db][4 * g4 + 2] * inv, acc_o[db][4 * g4 + 3] * inv)};
          *reinterpret_cast<u32x2*>(op + db * 32 + 8 * g4) = w;
        }
      if (a.lse && hf == 0)
        a.lse[((long long)i * a.H + h) * a.S + qi] = m_run * 0.69314718055994531f + logf(l_tot);
    }
  }
}

template <int DH>
cast_status_t launch_dh(AttnArgs a, hipStream_t stream) {
  a.n_qt = (a.S + 127) / 128;
  a.nblocks = a.n_a * a.H * a.n_qt;
  if (a.n0 == 0 && a.Bv >= kBK)
    hipLaunchKernelGGL((anchor_attn_kernel<DH, true>), dim3(a.nblocks), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((anchor_attn_kernel<DH, false>), dim3(a.nblocks), dim3(kThreads), 0, stream, a);
  return check_launch("anchor_attn");
}

}  // namespace

cast_status_t launch_anchor_attn(const void* q, const void* k_hist, const void* v_hist,
                                 const int32_t* idx, int k_eff, const void* k_cur,
                                 const void* v_cur, int n0, int n_a, int S, int H, int dh, int M,
                                 int Bv, float scale, void* out, float* lse_out,
                                 hipStream_t stream) {
  AttnArgs a{};
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k_hist);
  a.v = static_cast<const uint16_t*>(v_hist);
  a.idx = k_eff > 0 ? idx : nullptr;
  // keep every base pointer valid even for an empty segment (never dereferenced then)
  a.kc = static_cast<const uint16_t*>(n0 > 0 ? k_cur : k_hist);
  a.vc = static_cast<const uint16_t*>(n0 > 0 ? v_cur : v_hist);
  if (k_eff == 0) { a.k = a.kc; a.v = a.vc; }
  a.out = static_cast<uint16_t*>(out);
  a.lse = lse_out;
  a.n_a = n_a;
  a.S = S;
  a.H = H;
  a.M = M;
  a.Bv = Bv;
  a.n0 = n0;
  a.k_eff = k_eff;
  a.L = n0 + k_eff * Bv;
  a.bv_magic = ((1ull << 40) + (unsigned long long)Bv - 1) / (unsigned long long)Bv;
  a.sl2 = scale * 1.4426950408889634f;
  a.hist_bytes = k_eff > 0 ? (long long)M * Bv * H * dh * 2 : 0;
  a.cur_bytes = n0 > 0 ? (long long)n0 * H * dh * 2 : 0;
  switch (dh) {
    case 32: return launch_dh<32>(a, stream);
    case 64: return launch_dh<64>(a, stream);
    case 128: return launch_dh<128>(a, stream);
    default: return fail(CAST_ERR_UNSUPPORTED, "attn: dh %d", dh);
  }
}

}  // namespace cast
