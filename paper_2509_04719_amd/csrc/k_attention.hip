// Attention of a band's queries over the keys/values of the whole image,
// fresh for the band's tokens and stale (from the buffer) for all others
// (patch parallelism with stale activations, §II-B; Algorithm 1).
//
// bf16 path: a flash-style kernel on the matrix cores.  Each workgroup owns
// 128 queries of one (branch, head); each wave 32 of them.  Scores are formed
// transposed on v_mfma_f32_32x32x16_bf16, S^T = K Q^T, so that a lane owns one
// query column and the running max of the online softmax stays in-lane.
// O^T = V^T P^T runs on v_mfma_f32_16x16x32_bf16 (16-row tiles of O^T: d = 72
// pads to 80 rows, not 96); two lane swaps move the probabilities from the
// score layout into its B operand.
// K tiles ([64 keys][d], rows unpadded) and V^T tiles ([d][64 keys], 16-byte
// chunks XOR-swizzled by row) go global -> LDS with the direct-to-LDS load
// into a ring of four stages, one barrier per tile.  K rows are permuted in
// LDS (bits 2 and 3 of the row swapped) so that the 8 keys of each lane's P
// fragment are contiguous in natural key order.  When the head dimension is
// padded (d = 72 -> 80 rows of O^T), one padding row of V^T holds ones, so
// the PV product also accumulates the softmax denominator.  exp2 runs on
// v_exp_f32 with log2(e)/sqrt(d) folded into the exponent; the running max is
// set with headroom and raised lazily, tested after the exponentials by one
// bit of the packed bf16 probabilities, so O is rarely rescaled and no max is
// taken on the common path.  The loop
// runs over 32-key halves of a tile: the MFMAs of the next half's scores are
// issued between the current half's exponentials, then its PV MFMAs.  Built
// without IEEE NaN quieting, so the row max is plain v_max3_f32.
//
// fp32 path (and unsupported shapes): one thread per query, online softmax.
#include "common.h"
#include "kernels.h"

namespace orch {

namespace mfma_attn {
// BQ queries per workgroup (32 per wave), WPC workgroups per CU.  (256-query
// workgroups, one per CU, halve the K/V loads per CU but measured no faster,
// and slower where the query count is not a multiple of 256.)
constexpr int BQ = 128, BKV = 64, NSTAGE = 4;
constexpr int NW = BQ / 32, KW = NW / 2, NTHR = 64 * NW, WPC = 512 / NTHR;
// headroom of the running max: a raise puts it this far above the largest
// score so far, and the next raise comes when a score exceeds it by one, so
// the running max moves rarely (about once per 8 of score growth, log2 units)
constexpr float kLead = 7.0f;

template <int D>
struct Geo {
  static constexpr int NC = (D + 15) / 16;          // 16-dim chunks of S^T = K Q^T
  static constexpr int NS = 2 * NC;                 // MFMAs of one S^T tile
  static constexpr int DV = (D + 15) / 16 * 16;     // rows of O^T, padded to 16
  static constexpr int NT = DV / 16;                // 16-row tiles of O^T
  static constexpr bool ONES = DV > D;              // padding row D of V^T holds 1.0
  // d = 8 (mod 16): the upper half of the last 16-dim chunk is padding, where
  // K reads the constant (1, 1, 1, 0, ...) and Q carries -m_run split in three
  // bf16, so every score chain yields s - m_run from a zero accumulator
  static constexpr bool MCOL = D % 16 == 8;
  static constexpr int KROW = 2 * D;                // bytes per K row in LDS
  static constexpr int KCH = KROW / 16;             // 16-byte chunks per K row
  static constexpr bool KSWZ = KCH == 8;            // 128-byte rows: XOR swizzle
  static constexpr int K_BYTES = BKV * KROW;
  static constexpr int K_SPAN = (K_BYTES + 16 + 255) / 256 * 256;  // 16 constant bytes after K
  static constexpr int VROW = 2 * BKV;              // bytes per V^T row
  static constexpr int V_BYTES = D * VROW;
  static constexpr int STAGE = K_SPAN + V_BYTES;
  static constexpr int CONST_OFF = NSTAGE * STAGE;  // V^T rows [D, DV), shared by the stages
  static constexpr int DUMMY_OFF = CONST_OFF + (DV - D) * VROW;  // sink of padding loads
  static constexpr int LDS = DUMMY_OFF + 1024;
  static constexpr int K_LOADS = K_BYTES / 1024;    // 1 KB wave-level loads
  static constexpr int V_LOADS = V_BYTES / 1024;
  // the first KW waves load K, the others V^T, LPW loads each per tile;
  // slots past the tile's loads re-read a valid chunk into the sink, so
  // every wave counts the same number of loads
  static constexpr int LPW = (cmax(K_LOADS, V_LOADS) + KW - 1) / KW;
  static_assert(K_BYTES % 1024 == 0 && V_BYTES % 1024 == 0, "whole 1 KB loads");
  // 16 consecutive K rows at one 16-byte column must hit distinct 4-bank
  // groups: an odd number of chunks per row, or 8 chunks with the swizzle
  static_assert(KCH == 8 || KCH % 2 == 1, "K row layout");
  static_assert(WPC * LDS <= 160 * 1024, "workgroups per CU");
  static_assert((NSTAGE - 1) * LPW < 64, "loads in flight");
};

// LDS row rho of a K tile holds key kperm(rho): bits 2 and 3 swapped.  The
// S^T accumulator row 8g + 4h + r then belongs to key 16c + 8h + e for the
// P fragment (chunk c, element e) a lane with half h feeds to the PV MFMA,
// i.e. the 8 keys of a lane's fragment are contiguous and V^T stays in
// natural key order.
__device__ __forceinline__ int kperm(int rho) {
  return (rho & ~12) | ((rho & 4) << 1) | ((rho & 8) >> 1);
}

// word 3 of a raw buffer resource (gfx9: 32-bit data format, no swizzle)
constexpr int kBufWord3 = 0x00020000;

// Resource of a wave-uniform buffer; the base and size go through
// readfirstlane so the compiler keeps the descriptor in SGPRs.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, size_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  void* ub = reinterpret_cast<void*>(((uint64_t)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(ub, (short)0, __builtin_amdgcn_readfirstlane((int)bytes),
                                           kBufWord3);
}
}  // namespace mfma_attn

template <int D>
__global__ __launch_bounds__(mfma_attn::NTHR, mfma_attn::WPC) void attn_bf16_mfma_kernel(AttnParams p) {
  // the body uses device-only types (buffer resources); the host pass only
  // needs the launch stub
#if defined(__HIP_DEVICE_COMPILE__)
  using namespace mfma_attn;
  using G = Geo<D>;
  constexpr int NC = G::NC, NS = G::NS, NT = G::NT, LPW = G::LPW;

  extern __shared__ __attribute__((aligned(1024))) char smem[];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5;
  const int lc = lane & 31;
  // Work units: key tile k (64 keys) of query tile qt (128 queries) of
  // (branch, head), in the order (b, head, qt, k); workgroup w takes units
  // [w * per, (w + 1) * per).  Workgroups go round-robin over the 8 XCDs;
  // the ones of XCD x take the x-th contiguous eighth of the workers, so the
  // query tiles that read the same K/V share one L2.
  const int n_qt = (p.n_q + BQ - 1) / BQ;
  const int nkt = p.n_kv / BKV;                   // key tiles (launcher: n_kv % BKV == 0)
  const int units = n_qt * p.heads * p.B * nkt;
  const int T = gridDim.x;
  int w = blockIdx.x;
  if (w < T / 8 * 8) w = (w & 7) * __builtin_amdgcn_readfirstlane(T / 8) + (w >> 3);
  const int u_begin = w * p.per, u_end = min(u_begin + p.per, units);
  const int H = p.heads * D;
  const int fb = p.fresh_begin, nf = p.n_fresh;

  // constant LDS (never written by the tile loads): 16 bytes after the K
  // rows of every stage, bf16 (1, 1, 1, 0, 0, 0, 0, 0), the K side of the
  // max column; V^T rows [D, DV): row D ones, the rest zero
  for (int st = tid; st < NSTAGE * 4; st += NTHR) {
    const uint32_t one2 = 0x3F803F80u, one = 0x00003F80u;   // bf16 1.0 = 0x3F80
    reinterpret_cast<uint32_t*>(smem + (st >> 2) * G::STAGE + G::K_BYTES)[st & 3] =
        (st & 3) == 0 ? one2 : (st & 3) == 1 ? one : 0u;
  }
  {
    bf16* cpad = reinterpret_cast<bf16*>(smem + G::CONST_OFF);
    for (int i = tid; i < (G::DV - D) * BKV; i += NTHR) cpad[i] = (bf16)(i < BKV ? 1.0f : 0.0f);
  }

  // This wave's share of a tile's loads.  Waves [0, KW) load K: load j =
  // wave + KW i fills stage bytes [1024 j, +1024), lane slot s = 64 j + lane
  // is row s / KCH, physical chunk s % KCH.  Waves [KW, 2 KW) load V^T: load
  // j = wave - KW + KW i fills K_SPAN + 1024 j, row s / 8, physical chunk
  // s % 8, logical 8-key chunk = physical ^ ((row >> 1) & 7).  off: byte
  // offset of the lane's source from the tile's first key in the stale buffer
  // (the same for fresh K; fresh V^T rows have stride n_fresh).
  const bool kwave = wave < KW;
  const int wl = wave % KW;
  const int nload = kwave ? G::K_LOADS : G::V_LOADS;
  unsigned off[LPW];
#pragma unroll
  for (int i = 0; i < LPW; ++i) {
    const int j = min(wl + KW * i, nload - 1);
    const int sl = j * 64 + lane;
    if (kwave) {
      const int rho = sl / G::KCH, pc = sl % G::KCH;
      const int lch = G::KSWZ ? pc ^ ((rho >> 1) & 7) : pc;
      off[i] = (unsigned)(kperm(rho) * D + lch * 8) * 2u;
    } else {
      const int d = sl >> 3, lch = (sl & 7) ^ ((d >> 1) & 7);
      off[i] = (unsigned)(d * p.n_kv + lch * 8) * 2u;
    }
  }
  // V^T row of load slot i (V waves)
  auto vrow = [&](int i) { return (min(wl + KW * i, nload - 1) * 64 + lane) >> 3; };
  auto dst_of = [&](int st, int i) -> ORCH_LDS void* {
    const int j = wl + KW * i;
    if (j >= nload) return (ORCH_LDS void*)(smem + G::DUMMY_OFF);
    return (ORCH_LDS void*)(smem + st * G::STAGE + (kwave ? 0 : G::K_SPAN) + j * 1024);
  };
  // state of the current segment's (branch, head): K/V bases, their buffer
  // resources (out-of-range reads return zero), this lane's Q fragments
  const int fn = nf > 0 ? p.fresh_n : p.n_kv;     // token extent of the fresh buffer
  const bf16 *ks, *vs, *kf, *vf;
  __amdgpu_buffer_rsrc_t rks, rvs, rkf, rvf;
  bf16x8 qf[NC];
  auto issue = [&](int n0, int st) {
    const bool all_stale = n0 + BKV <= fb || n0 >= fb + nf;
    const bool all_fresh = n0 >= fb && n0 + BKV <= fb + nf;
    if (all_stale) {
      const __amdgpu_buffer_rsrc_t r = kwave ? rks : rvs;
      const unsigned so = __builtin_amdgcn_readfirstlane((unsigned)n0 * (kwave ? 2 * D : 2));
#pragma unroll
      for (int i = 0; i < LPW; ++i) __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst_of(st, i), 16, off[i], so, 0, 0);
    } else if (all_fresh) {
      const __amdgpu_buffer_rsrc_t r = kwave ? rkf : rvf;
      const unsigned so = __builtin_amdgcn_readfirstlane((unsigned)(n0 - fb) * (kwave ? 2 * D : 2));
#pragma unroll
      for (int i = 0; i < LPW; ++i) {
        const unsigned o = kwave ? off[i] : off[i] - (unsigned)(vrow(i) * (p.n_kv - fn)) * 2u;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst_of(st, i), 16, o, so, 0, 0);
      }
    } else {
      // a tile across the band edge: each lane loads from the buffer its 8
      // keys live in (8-key groups are all fresh or all stale: fb, nf % 8 ==
      // 0), the two buffer loads under complementary lane masks.  A wave may
      // then count two loads for one slot; the waits below only need at least
      // LPW per tile, so they wait longer, never shorter.
      const unsigned so = __builtin_amdgcn_readfirstlane((unsigned)n0 * (kwave ? 2 * D : 2));
#pragma unroll
      for (int i = 0; i < LPW; ++i) {
        const int n = n0 + (kwave ? (int)(off[i] / 2) / D : (int)(off[i] / 2) - vrow(i) * p.n_kv);
        if ((unsigned)(n - fb) < (unsigned)nf) {
          const int o = kwave ? (int)off[i] + (n0 - fb) * 2 * D
                              : (int)off[i] - vrow(i) * (p.n_kv - fn) * 2 + (n0 - fb) * 2;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(kwave ? rkf : rvf, dst_of(st, i), 16, (unsigned)o, 0, 0, 0);
        } else {
          __builtin_amdgcn_raw_ptr_buffer_load_lds(kwave ? rks : rvs, dst_of(st, i), 16, off[i], so, 0, 0);
        }
      }
    }
  };
  // wait until at most `tiles` tiles of this wave's loads are in flight
  auto wait_tiles = [&](int tiles) {
    if (tiles <= 0) wait_vmcnt<0>();
    else if (tiles == 1) wait_vmcnt<LPW>();
    else wait_vmcnt<2 * LPW>();
  };

  // fragment read offsets: K row sub*32 + lc, logical chunk 2c + h (A of the
  // 32x32x16 MFMA: row lane & 31, k 8 (lane >> 5) .. +8); V^T row 16 t + r16,
  // logical chunk 4 psub + (lane >> 4) (A of the 16x16x32 MFMA: row lane & 15,
  // k 8 (lane >> 4) .. +8; the swizzle depends on r16 only).  V^T rows >= D
  // are the shared constant rows.
  // (unswizzled rows: one base, the chunks at immediate offsets 32 c)
  int k_rd[G::KSWZ ? NC : 1];
#pragma unroll
  for (int c = 0; c < (G::KSWZ ? NC : 1); ++c)
    k_rd[c] = lc * G::KROW + (G::KSWZ ? ((2 * c + h) ^ ((lc >> 1) & 7)) : (2 * c + h)) * 16;
  const int r16 = lane & 15, g16 = lane >> 4;
  int v_rd[2];
#pragma unroll
  for (int ps = 0; ps < 2; ++ps) v_rd[ps] = r16 * G::VROW + ((4 * ps + g16) ^ ((r16 >> 1) & 7)) * 16;
  const bool last_in_pad = (NT - 1) * 16 + r16 >= D;   // row of the last O^T tile is padding
  // the last K chunk of half sub: the max column's constant on the h = 1 lanes
  int k_last[2];
#pragma unroll
  for (int sub = 0; sub < 2; ++sub)
    k_last[sub] = G::MCOL && h ? G::K_BYTES
                               : sub * 32 * G::KROW + (G::KSWZ ? k_rd[NC - 1] : k_rd[0] + 32 * (NC - 1));

  const float scale = 1.4426950408889634f / sqrtf((float)D);  // log2(e) / sqrt(d)
  float m_run, l_run;
  // O^T tile t (rows 16 t .. +16) of the queries 16 j + (lane & 15) is the
  // 4-float accumulator f = 2 t + j, elements 4 (f % 4) .. +4 of oo[f / 4].
  // (As separate 4-float values the register allocator moved every one of
  // them between two register sets each half-step: 65 copies per tile and
  // 54 more registers; held in 16-float tuples they stay in place.)
  f32x16 oo[(2 * NT + 3) / 4];
  auto oget = [&](int t, int j) __attribute__((always_inline)) {
    const int f = 2 * t + j;
    f32x4 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = oo[f / 4][4 * (f % 4) + i];
    return r;
  };
  auto oset = [&](int t, int j, const f32x4& r) __attribute__((always_inline)) {
    const int f = 2 * t + j;
#pragma unroll
    for (int i = 0; i < 4; ++i) oo[f / 4][4 * (f % 4) + i] = r[i];
  };
  f32x16 negm;   // without the max column: -m_run in every element, the input of each score chain
  const f32x16 zero16 = {};
  // -m_run into the max column of Q (h = 1 lanes, last chunk): three bf16
  // whose sum is exactly -m_run (each takes the next 8 significant bits by
  // truncation; any fp32 splits so)
  auto set_mcol = [&]() {
    const float a0 = -m_run;
    const float b0 = __uint_as_float(__float_as_uint(a0) & 0xFFFF0000u);
    const float r0 = a0 - b0;
    const float b1 = __uint_as_float(__float_as_uint(r0) & 0xFFFF0000u);
    const float b2 = r0 - b1;
    if (h) {
      qf[NC - 1][0] = (bf16)b0;
      qf[NC - 1][1] = (bf16)b1;
      qf[NC - 1][2] = (bf16)b2;
    }
  };
  // first accumulator input of a score chain
  auto chain_in = [&]() -> const f32x16& {
    if constexpr (G::MCOL) return zero16;
    else return negm;
  };

  // K fragments of half `sub` (keys [32 sub, +32)) of the tile in stage st
  auto k_frags = [&](int st, int sub, bf16x8(&kf_)[NC]) {
    const char* sk = smem + st * G::STAGE + sub * 32 * G::KROW;
#pragma unroll
    for (int c = 0; c < NC - 1; ++c)
      kf_[c] = *reinterpret_cast<const bf16x8*>(sk + (G::KSWZ ? k_rd[c] : k_rd[0] + 32 * c));
    kf_[NC - 1] = *reinterpret_cast<const bf16x8*>(smem + st * G::STAGE + (sub ? k_last[1] : k_last[0]));
  };
  // V^T fragment of O^T tile tt, keys of half ps, of the tile in stage st
  auto v_frag = [&](int st, int tt, int ps) {
    const char* src = (tt == NT - 1 && last_in_pad)
                          ? smem + G::CONST_OFF + (tt * 16 + r16 - D) * G::VROW + (v_rd[ps] - r16 * G::VROW)
                          : smem + st * G::STAGE + G::K_SPAN + tt * 16 * G::VROW + v_rd[ps];
    return *reinterpret_cast<const bf16x8*>(src);
  };
  // P^T of a 32-key half from the score layout (16-key chunk ci, lane half h:
  // keys 16 ci + 8 h .. +8 of query lane & 31) into the B layout of the
  // 16x16x32 MFMA (pq[j], lane l: keys 8 (l >> 4) .. +8 of query 16 j +
  // (l & 15)).  In 16-lane rows, chunk 0 = (a0 a1 a2 a3) and chunk 1 =
  // (b0 b1 b2 b3): the 32-lane swap gives (a0 a1 b0 b1) and (a2 a3 b2 b3), the
  // 16-lane swap then (a0 a2 b0 b2) = queries 0-15 and (a1 a3 b1 b3) = 16-31.
  auto p_swap = [&](bf16x8(&pp)[2]) __attribute__((always_inline)) {
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 x = __builtin_bit_cast(u32x4, pp[0]), y = __builtin_bit_cast(u32x4, pp[1]);
    u32x4 q0, q1;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const auto r = __builtin_amdgcn_permlane32_swap(x[i], y[i], false, false);
      const auto t = __builtin_amdgcn_permlane16_swap(r[0], r[1], false, false);
      q0[i] = t[0];
      q1[i] = t[1];
    }
    pp[0] = __builtin_bit_cast(bf16x8, q0);
    pp[1] = __builtin_bit_cast(bf16x8, q1);
  };

  // the largest of a query's 32 scores (its two lane halves)
  auto query_max = [&](const f32x16& v) {
    float mx = fmaxf(fmaxf(v[0], v[1]), v[2]);
#pragma unroll
    for (int r = 3; r < 15; r += 2) mx = fmaxf(fmaxf(mx, v[r]), v[r + 1]);
    return max_xhalf(fmaxf(mx, v[15]));
  };
  // -m_run into the score chains' input (max column or accumulator)
  auto m_changed = [&]() {
    if constexpr (G::MCOL) {
      set_mcol();
    } else {
#pragma unroll
      for (int r = 0; r < 16; ++r) negm[r] = -m_run;
    }
  };

  // One 32-key half of the stream of key tiles.  sc: S^T of keys [32 sub,
  // +32) of the tile in stage st.  Its exponentials are interleaved with the
  // MFMAs of the next half's scores (NEXT: K fragments of stage nst, half
  // nsub, into sn) and of the previous half's O^T += V^T P^T (probabilities
  // pp in the score layout, V^T of stage pst, half psub), so a wave keeps its
  // matrix core busy through the softmax.  This half's probabilities go to pc.
  auto step = [&](auto next_c, bool start, int st, int sub, f32x16& sc, int nst, int nsub,
                  f32x16& sn, int pst, int psub, bf16x8(&pp)[2], bf16x8(&pc)[2]) {
    constexpr bool NEXT = decltype(next_c)::value;
    // online softmax over this lane's query column.  Q carries log2(e)/sqrt(d)
    // and every score chain subtracts m_run (through the max column, else as
    // the accumulator input), so sc holds s - m_run and the probability is
    // exp2(sc) with nothing in between.
    // The running max m_run is a whole number: a segment's first half sets it
    // kLead above its largest score; later halves compute their probabilities
    // first and test them afterwards with one bit (any probability >= 2), so
    // no max is taken while the probabilities stay below 2.  When one reaches
    // 2, the half's scores are lowered by a whole d (to kLead below the new
    // max), its probabilities recomputed and O scaled by 2^-d.  The fragment
    // reads go first, in order of use; the lane swaps cover their latency.
    bf16x8 vp[NT];
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) vp[tt] = v_frag(pst, tt, psub);
    bf16x8 kn[NC];
    if constexpr (NEXT) k_frags(nst, nsub, kn);
    p_swap(pp);   // pp[j]: queries 16 j .. +16
    if (start) {
      // m_run is zero here, O and the pending probabilities too
      const float d = ceilf(query_max(sc)) + kLead;
      m_run = d;
#pragma unroll
      for (int r = 0; r < 16; ++r) sc[r] -= d;
      m_changed();
    }
    __builtin_amdgcn_sched_barrier(0);
    // the MFMA-dense part runs at raised wave priority: the two waves sharing a
    // SIMD then fall out of step, one in its softmax while the other issues
    // MFMAs (measured 3-4% faster than equal priorities)
    __builtin_amdgcn_s_setprio(1);
    float psum = 0.0f;
    // per 16-key chunk ci: NM MFMAs (PV of query block ci and S alternating,
    // PV first) in groups, each followed by its share of the chunk's 4 pairs
    // of exponentials; a scheduling fence after each group keeps the order
    static_for<0, 2>([&](auto cc) {
      constexpr int ci = decltype(cc)::value;
      constexpr int c0 = ci * NC / 2, c1 = (ci + 1) * NC / 2;
      constexpr int NSM = NEXT ? c1 - c0 : 0, NM = NSM + NT, NB = cmin(NSM, NT);
      static_for<0, NM>([&](auto gc) {
        constexpr int g = decltype(gc)::value;
        constexpr bool pv = g < 2 * NB ? g % 2 == 0 : NT > NSM;
        constexpr int idx = g < 2 * NB ? g / 2 : g - NB;
        if constexpr (pv)
          oset(idx, ci, __builtin_amdgcn_mfma_f32_16x16x32_bf16(vp[idx], pp[ci], oget(idx, ci), 0, 0, 0));
        else
          sn = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kn[c0 + idx], qf[c0 + idx],
                                                      c0 + idx == 0 ? chain_in() : sn, 0, 0, 0);
        static_for<g * 4 / NM, (g + 1) * 4 / NM>([&](auto pc_) {
          constexpr int pr = decltype(pc_)::value;
#pragma unroll
          for (int e = 2 * pr; e < 2 * pr + 2; ++e) {
            const int r = 4 * (2 * ci + (e >> 2)) + (e & 3);
            const float pv_ = __builtin_amdgcn_exp2f(sc[r]);
            if constexpr (!G::ONES) psum += pv_;
            pc[ci][e] = (bf16)pv_;
          }
        });
        __builtin_amdgcn_sched_barrier(0);
      });
      // the probabilities are consumed one half later (by the next step or
      // after the loop); this empty use keeps their exponentials here, between
      // the MFMAs, instead of sunk into the next block
      asm volatile("" ::"v"(pc[ci]));
    });
    __builtin_amdgcn_s_setprio(0);
    // any probability >= 2 (or not finite): bf16 exponent bit 7 set
    float alpha = 1.0f;
    {
      typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
      const u32x4 a = __builtin_bit_cast(u32x4, pc[0]), b = __builtin_bit_cast(u32x4, pc[1]);
      const unsigned w = a[0] | a[1] | a[2] | a[3] | b[0] | b[1] | b[2] | b[3];
      if (__builtin_expect(__any((w & 0x40004000u) != 0u), 0)) {
        const float mx = query_max(sc);
        const float d = mx >= 1.0f ? ceilf(mx) + kLead : 0.0f;
        alpha = ldexpf(1.0f, -(int)fminf(d, 160.0f));
        m_run += d;
#pragma unroll
        for (int r = 0; r < 16; ++r) sc[r] -= d;
        // the next half's scores were formed with the old m_run
        if constexpr (NEXT) {
#pragma unroll
          for (int r = 0; r < 16; ++r) sn[r] -= d;
        }
        m_changed();
        psum = 0.0f;
#pragma unroll
        for (int ci = 0; ci < 2; ++ci)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float pv_ = __builtin_amdgcn_exp2f(sc[4 * (2 * ci + (e >> 2)) + (e & 3)]);
            if constexpr (!G::ONES) psum += pv_;
            pc[ci][e] = (bf16)pv_;
          }
        // O^T holds queries 16 j + (lane & 15); its PV products so far used
        // the old m_run
        float aj[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) aj[j] = __shfl(alpha, 16 * j + r16, kWave);
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int tt = 0; tt < NT; ++tt)
#pragma unroll
            for (int r = 0; r < 4; ++r) oo[(2 * tt + j) / 4][4 * ((2 * tt + j) % 4) + r] *= aj[j];   // oget(tt, j) *= aj[j]
      }
    }
    if constexpr (!G::ONES) l_run = l_run * alpha + psum;
  };

  // segments: key tiles [a, bnd) of query tile `tile`, last tile of the
  // range first.  With at most two segments (a range shorter than a tile),
  // every workgroup then starts at key tile 0 and, in its second segment,
  // reads key tile tau + nkt - per at time tau: the workgroups of one head
  // sweep its K/V in step and share each tile in L2.  (The divisions run on
  // the VALU; readfirstlane keeps the segment's indices, and the loop
  // control built on them, in SGPRs.)
  const int tile_first = __builtin_amdgcn_readfirstlane(u_begin / nkt);
  for (int ue = u_end; ue > u_begin;) {
    const int tile = __builtin_amdgcn_readfirstlane((ue - 1) / nkt);
    const int a = max(u_begin - tile * nkt, 0), bnd = ue - tile * nkt;
    const bool first = ue == u_end;                 // first segment processed
    ue = tile * nkt + a;
    const int pair = __builtin_amdgcn_readfirstlane(tile / n_qt), qt = tile - pair * n_qt;
    const int b = __builtin_amdgcn_readfirstlane(pair / p.heads), head = pair - b * p.heads;
    // (readfirstlane: the compiler otherwise keeps these two in VGPRs, and
    // the per-tile load issue and waits become exec-masked branches; in
    // SGPRs they are scalar compares, 2.5% faster)
    const int q0 = qt * BQ, kv0 = __builtin_amdgcn_readfirstlane(a * BKV),
              NIT = __builtin_amdgcn_readfirstlane(bnd - a);
    if (!first) lds_barrier();   // every wave is done with the previous segment's stages
    const bf16* qbase = reinterpret_cast<const bf16*>(p.q) + ((size_t)b * p.heads + head) * p.n_q * D;
    ks = reinterpret_cast<const bf16*>(p.kv_stale) + b * p.stale_bs + (size_t)head * p.n_kv * D;
    vs = reinterpret_cast<const bf16*>(p.kv_stale) + b * p.stale_bs + (size_t)p.n_kv * H +
         (size_t)head * D * p.n_kv;
    kf = ks;
    vf = vs;
    if (nf > 0) {
      kf = reinterpret_cast<const bf16*>(p.kv_fresh) + b * p.fresh_bs + ((size_t)head * fn + p.fresh_off) * D;
      vf = reinterpret_cast<const bf16*>(p.kv_fresh) + b * p.fresh_bs + (size_t)fn * H +
           (size_t)head * D * fn + p.fresh_off;
    }
    rks = buffer_rsrc(ks, (size_t)p.n_kv * D * 2);
    rvs = buffer_rsrc(vs, (size_t)p.n_kv * D * 2);
    rkf = buffer_rsrc(kf, (size_t)(nf > 0 ? nf : p.n_kv) * D * 2);
    rvf = buffer_rsrc(vf, ((size_t)(D - 1) * fn + (nf > 0 ? nf : p.n_kv)) * 2);
    // this lane's query (B operand of S^T = K Q^T): Q[q][c*16 + 8h .. +8]
    const int qrow = min(q0 + wave * 32 + lc, p.n_q - 1);
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int d0 = c * 16 + h * 8;
      if (d0 < D) {
        const bf16x8 qv = *reinterpret_cast<const bf16x8*>(qbase + (size_t)qrow * D + d0);
        if (p.q_scaled) {
          qf[c] = qv;
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) qf[c][e] = (bf16)((float)qv[e] * scale);
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[c][e] = (bf16)0.0f;
      }
    }
    m_run = 0.0f;
    if constexpr (!G::MCOL) {
#pragma unroll
      for (int r = 0; r < 16; ++r) negm[r] = 0.0f;
    }
    l_run = 0.0f;
#pragma unroll
    for (int k = 0; k < (2 * NT + 3) / 4; ++k)
#pragma unroll
      for (int r = 0; r < 16; ++r) oo[k][r] = 0.0f;

#pragma unroll
    for (int s = 0; s < NSTAGE - 1; ++s)
      if (s < NIT) issue(kv0 + s * BKV, s);
    wait_tiles(min(NIT - 1, NSTAGE - 2));
    lds_barrier();

    // scores ping-pong between s0 (first halves) and s1 (second halves)
    f32x16 s0, s1;
    bf16x8 kn[NC];
    k_frags(0, 0, kn);   // the first half's scores
    s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kn[0], qf[0], chain_in(), 0, 0, 0);
#pragma unroll
    for (int c = 1; c < NC; ++c) s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kn[c], qf[c], s0, 0, 0, 0);

    // probabilities of the previous and the current half, ping-pong; the
    // first half's "previous" is zero against resident V^T rows
    bf16x8 pa[2], pb[2];
#pragma unroll
    for (int ci = 0; ci < 2; ++ci)
#pragma unroll
      for (int e = 0; e < 8; ++e) pa[ci][e] = (bf16)0.0f;
    int t = 0;
    for (; t + 1 < NIT; ++t) {
      const int st = t % NSTAGE;
      const int pst = t == 0 ? st : (t + NSTAGE - 1) % NSTAGE;
      step(std::true_type{}, t == 0, st, 0, s0, st, 1, s1, pst, t == 0 ? 0 : 1, pa, pb);
      // tile t+1 resident; stage (t-1) % NSTAGE is free for tile t+3
      wait_tiles(t + 2 < NIT ? 1 : 0);
      lds_barrier();
      if (t + NSTAGE - 1 < NIT) issue(kv0 + (t + NSTAGE - 1) * BKV, (t + NSTAGE - 1) % NSTAGE);
      step(std::true_type{}, false, st, 1, s1, (t + 1) % NSTAGE, 0, s0, st, 0, pb, pa);
    }
    {
      const int st = t % NSTAGE;
      const int pst = t == 0 ? st : (t + NSTAGE - 1) % NSTAGE;
      step(std::true_type{}, t == 0, st, 0, s0, st, 1, s1, pst, t == 0 ? 0 : 1, pa, pb);
      step(std::false_type{}, false, st, 1, s1, 0, 0, s0, st, 0, pb, pa);
      // the last half's PV
      bf16x8 vp[NT];
#pragma unroll
      for (int tt = 0; tt < NT; ++tt) vp[tt] = v_frag(st, tt, 1);
      p_swap(pa);
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int tt = 0; tt < NT; ++tt)
          oset(tt, j, __builtin_amdgcn_mfma_f32_16x16x32_bf16(vp[tt], pa[j], oget(tt, j), 0, 0, 0));
    }

    // softmax denominator of query 16 j + (lane & 15): the ones row D of O^T
    // (tile D / 16, register (D % 16) % 4 of the lanes 16 ((D % 16) / 4) ..
    // +16), or the running sums of the query's two lane halves
    float lj[2];
    if constexpr (G::ONES) {
      constexpr int TR = D / 16, RG = (D % 16) / 4, RR = (D % 16) % 4;
#pragma unroll
      for (int j = 0; j < 2; ++j) lj[j] = __shfl(oget(TR, j)[RR], 16 * RG + r16, kWave);
    } else {
      const float lq = l_run + __shfl_xor(l_run, 32, kWave);
#pragma unroll
      for (int j = 0; j < 2; ++j) lj[j] = __shfl(lq, 16 * j + r16, kWave);
    }
    // a whole query tile goes to the output; the part of a cut one to this
    // workgroup's slot (2w: the first tile of its range, 2w + 1: the last) as
    // O_s / l_s in bf16 with (max, sum), for the merge.  A lane holds dims
    // 16 t + 4 (lane >> 4) .. +4 of queries 16 j + (lane & 15).
    const bool whole = a == 0 && bnd == nkt;
    const int slot = 2 * w + (tile == tile_first ? 0 : 1);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int ql = wave * 32 + 16 * j + r16, q = q0 + ql;
      const float inv = 1.0f / lj[j];
      if (q < p.n_q) {
        bf16* orow = whole ? reinterpret_cast<bf16*>(p.out) + ((size_t)b * p.n_q + q) * H + head * D
                           : reinterpret_cast<bf16*>(p.part_o) + ((size_t)slot * BQ + ql) * D;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const int d = 16 * t + 4 * g16;
          if (d < D) {
            bf16x4 v;
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] = (bf16)(oget(t, j)[i] * inv);
            *reinterpret_cast<bf16x4*>(orow + d) = v;
          }
        }
      }
    }
    // (max, sum) of the query lane & 31 of the score layout, whose sum is
    // lj[(lane & 31) >> 4] here
    const int ql = wave * 32 + lc;
    if (!whole && h == 0 && q0 + ql < p.n_q)
      p.part_ml[(size_t)slot * BQ + ql] = make_float2(m_run, lc >> 4 ? lj[1] : lj[0]);
  }
#endif
}

// Merge of the parts of the query tiles cut between workgroups.  Part s
// holds O_s / l_s with its running max m_s and sum l_s (log2 domain of the
// kernel above); O = sum_s 2^(m_s - m) l_s (O_s / l_s) / sum_s 2^(m_s - m) l_s
// with m = max_s m_s.  One thread per 8 channels of a query; grid (chunk
// groups, query tiles).  The parts are taken four at a time with their loads
// issued together (a tile is cut into two or three parts in the common
// case), merged online.  Tiles computed whole return at once.  A tile's
// 128 x D / 8 threads fill whole workgroups (three of 384 for d = 72).
template <int D>
struct MergeGeo {
  static constexpr int CPQ = D / 8;                // 16-byte chunks per query
  static constexpr int THREADS = mfma_attn::BQ * CPQ % 384 == 0 ? 384 : 256;
  static constexpr int BLOCKS = (mfma_attn::BQ * CPQ + THREADS - 1) / THREADS;
};

template <int D>
__global__ __launch_bounds__(MergeGeo<D>::THREADS) void attn_merge_kernel(AttnParams p) {
  using namespace mfma_attn;
  constexpr int CPQ = MergeGeo<D>::CPQ;
  const int nkt = p.n_kv / BKV, n_qt = (p.n_q + BQ - 1) / BQ;
  const int tile = blockIdx.y;
  const int w0 = tile * nkt / p.per, w1 = (tile * nkt + nkt - 1) / p.per;
  if (w0 == w1) return;
  const int i = blockIdx.x * MergeGeo<D>::THREADS + threadIdx.x;
  const int ql = i / CPQ, c = i - ql * CPQ;
  const int qt = tile % n_qt, pair = tile / n_qt;
  const int q = qt * BQ + ql;
  if (ql >= BQ || q >= p.n_q) return;
  const int head = pair % p.heads, b = pair / p.heads;
  const bf16* part = reinterpret_cast<const bf16*>(p.part_o);
  float m = -1e30f, den = 0.0f, num[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  for (int wb = w0; wb <= w1; wb += 4) {
    float2 ml[4];
    bf16x8 v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int w = wb + k;
      if (w <= w1) {
        const int slot = 2 * w + (w * p.per / nkt == tile ? 0 : 1);
        ml[k] = p.part_ml[(size_t)slot * BQ + ql];
        v[k] = *reinterpret_cast<const bf16x8*>(part + ((size_t)slot * BQ + ql) * D + c * 8);
      } else {
        ml[k] = make_float2(-1e30f, 0.0f);
#pragma unroll
        for (int e = 0; e < 8; ++e) v[k][e] = (bf16)0.0f;
      }
    }
    float mc = m;
#pragma unroll
    for (int k = 0; k < 4; ++k) mc = fmaxf(mc, ml[k].x);
    const float f = __builtin_amdgcn_exp2f(m - mc);
    m = mc;
    den *= f;
#pragma unroll
    for (int e = 0; e < 8; ++e) num[e] *= f;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float wt = __builtin_amdgcn_exp2f(ml[k].x - m) * ml[k].y;
      den += wt;
#pragma unroll
      for (int e = 0; e < 8; ++e) num[e] = fmaf(wt, (float)v[k][e], num[e]);
    }
  }
  const float inv = 1.0f / den;
  bf16x8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = (bf16)(num[e] * inv);
  *reinterpret_cast<bf16x8*>(reinterpret_cast<bf16*>(p.out) + ((size_t)b * p.n_q + q) * p.heads * D +
                             head * D + c * 8) = r;
}

// ---------------------------------------------------------------------------
// SIMT attention: one thread per (branch, head, query).
template <typename T, int D>
__global__ __launch_bounds__(64) void attn_simt_kernel(AttnParams p) {
  const int q = blockIdx.x * 64 + threadIdx.x;
  const int head = blockIdx.y;
  const int b = blockIdx.z;
  if (q >= p.n_q) return;
  const int H = p.heads * D;
  const T* qv = reinterpret_cast<const T*>(p.q) + (((size_t)b * p.heads + head) * p.n_q + q) * D;
  const T* ks = reinterpret_cast<const T*>(p.kv_stale) + b * p.stale_bs + (size_t)head * p.n_kv * D;
  const T* vs = reinterpret_cast<const T*>(p.kv_stale) + b * p.stale_bs + (size_t)p.n_kv * H +
                (size_t)head * D * p.n_kv;
  const T* kf = nullptr;
  const T* vf = nullptr;
  if (p.n_fresh > 0) {
    kf = reinterpret_cast<const T*>(p.kv_fresh) + b * p.fresh_bs +
         ((size_t)head * p.fresh_n + p.fresh_off) * D;
    vf = reinterpret_cast<const T*>(p.kv_fresh) + b * p.fresh_bs + (size_t)p.fresh_n * H +
         (size_t)head * D * p.fresh_n + p.fresh_off;
  }
  // scores in the log2 domain: q carries log2(e)/sqrt(d) when p.q_scaled
  float qr[D], acc[D];
  const float scale = p.q_scaled ? 1.0f : 1.4426950408889634f / sqrtf((float)D);
#pragma unroll
  for (int d = 0; d < D; ++d) {
    qr[d] = to_f<T>(qv[d]) * scale;
    acc[d] = 0.0f;
  }
  float m = -INFINITY, l = 0.0f;
  for (int n = 0; n < p.n_kv; ++n) {
    const int f = n - p.fresh_begin;
    const bool fresh = (unsigned)f < (unsigned)p.n_fresh;
    const T* kr = fresh ? kf + (size_t)f * D : ks + (size_t)n * D;
    float s = 0.0f;
#pragma unroll
    for (int d = 0; d < D; ++d) s = fmaf(qr[d], to_f<T>(kr[d]), s);
    const float mn = fmaxf(m, s);
    const float a = exp2f(m - mn);
    const float e = exp2f(s - mn);
    l = l * a + e;
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const float v = fresh ? to_f<T>(vf[(size_t)d * p.fresh_n + f]) : to_f<T>(vs[(size_t)d * p.n_kv + n]);
      acc[d] = fmaf(acc[d], a, e * v);
    }
    m = mn;
  }
  T* o = reinterpret_cast<T*>(p.out) + ((size_t)b * p.n_q + q) * H + head * D;
  const float inv = 1.0f / l;
#pragma unroll
  for (int d = 0; d < D; ++d) o[d] = from_f<T>(acc[d] * inv);
}

// ---------------------------------------------------------------------------
bool attention_uses_mfma(int d, int n_kv, int dtype) {
  return dtype == kBF16 && (d == 64 || d == 72) && n_kv % mfma_attn::BKV == 0;
}

template <typename T>
static hipError_t launch_simt(const AttnParams& p, hipStream_t s) {
  dim3 grid(ceil_div(p.n_q, 64), p.heads, p.B);
  switch (p.d) {
    case 32: hipLaunchKernelGGL((attn_simt_kernel<T, 32>), grid, dim3(64), 0, s, p); break;
    case 64: hipLaunchKernelGGL((attn_simt_kernel<T, 64>), grid, dim3(64), 0, s, p); break;
    case 72: hipLaunchKernelGGL((attn_simt_kernel<T, 72>), grid, dim3(64), 0, s, p); break;
    case 80: hipLaunchKernelGGL((attn_simt_kernel<T, 80>), grid, dim3(64), 0, s, p); break;
    case 96: hipLaunchKernelGGL((attn_simt_kernel<T, 96>), grid, dim3(64), 0, s, p); break;
    case 128: hipLaunchKernelGGL((attn_simt_kernel<T, 128>), grid, dim3(64), 0, s, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Work plan.  Units are (branch, head, query tile, key tile).  Whole query
// tiles per workgroup leave CUs idle when the tile count is not close to a
// multiple of 512 (two workgroups per CU); with a workspace, every workgroup
// takes per = ceil(units / 512) units instead, cutting query tiles between
// workgroups, when that shortens the longest workgroup by more than
// kCutTiles key tiles: a workgroup whose range crosses a tile boundary
// starts a second segment (its queries and first key tiles loaded again),
// and the parts go through the merge kernel, together about 15 us on
// MI355X at 1.2 us a key tile.  (At DiT-XL/2 1024px, 40% band, 52 key tiles
// per workgroup cut against 64 whole measured 77.0 against 75.3 us in the
// step; at 25% and 65% the cut saves 9 and 22 us.)
struct AttnPlan {
  int per, workers;
  size_t ws_bytes;   // parts of cut tiles; 0 when tiles stay whole
};

static AttnPlan plan_attention(int B, int heads, int n_q, int n_kv, int d) {
  constexpr int kSlots = 256 * mfma_attn::WPC;
  const int nkt = n_kv / mfma_attn::BKV;
  const int tiles = ceil_div(n_q, mfma_attn::BQ) * heads * B;
  const long long units = (long long)tiles * nkt;
  const int per = (int)((units + kSlots - 1) / kSlots);
  const long long whole_longest = (long long)nkt * ceil_div(tiles, kSlots);
  constexpr int kCutTiles = 12;
  if (per % nkt == 0 || per + kCutTiles >= whole_longest) return {nkt, tiles, 0};
  const int workers = (int)((units + per - 1) / per);
  const size_t parts = (size_t)2 * workers * mfma_attn::BQ;
  return {per, workers, (parts * d * 2 + 255) / 256 * 256 + parts * sizeof(float2)};
}

size_t attention_workspace_bytes(int B, int heads, int n_q, int n_kv, int d, int dtype) {
  if (n_q <= 0 || B <= 0 || heads <= 0 || !attention_uses_mfma(d, n_kv, dtype)) return 0;
  return plan_attention(B, heads, n_q, n_kv, d).ws_bytes;
}

static bool aligned16(const void* ptr) { return ((uintptr_t)ptr & 15) == 0; }

template <int D>
static void launch_mfma(dim3 grid, const AttnParams& p, hipStream_t s) {
  constexpr int lds = mfma_attn::Geo<D>::LDS;
  auto kern = attn_bf16_mfma_kernel<D>;
  static bool attr = [&] {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                              hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    return true;
  }();
  (void)attr;
  hipLaunchKernelGGL(kern, grid, dim3(mfma_attn::NTHR), lds, s, p);
}

hipError_t launch_attention(const AttnParams& p0, int dtype, hipStream_t s) {
  if (p0.n_q <= 0) return hipSuccess;
  AttnParams p = p0;
  // the MFMA kernel moves 16-byte chunks of Q, K and V^T (8 keys of V^T at a
  // time, all fresh or all stale)
  const bool aligned = p.fresh_begin % 8 == 0 && p.n_fresh % 8 == 0 && aligned16(p.q) &&
                       aligned16(p.kv_stale) && p.stale_bs % 8 == 0 &&
                       (p.n_fresh == 0 || (aligned16(p.kv_fresh) && p.fresh_bs % 8 == 0 &&
                                           p.fresh_n % 8 == 0 && p.fresh_off % 8 == 0));
  if (attention_uses_mfma(p.d, p.n_kv, dtype) && aligned) {
    const AttnPlan plan = plan_attention(p.B, p.heads, p.n_q, p.n_kv, p.d);
    const int nkt = p.n_kv / mfma_attn::BKV;
    const int tiles = ceil_div(p.n_q, mfma_attn::BQ) * p.heads * p.B;
    const bool cut = plan.ws_bytes > 0 && p.ws && p.ws_bytes >= plan.ws_bytes;
    p.per = cut ? plan.per : nkt;
    p.workers = cut ? plan.workers : tiles;
    p.part_o = nullptr;
    p.part_ml = nullptr;
    if (cut) {
      const size_t parts = (size_t)2 * p.workers * mfma_attn::BQ;
      p.part_o = p.ws;
      p.part_ml = reinterpret_cast<float2*>(reinterpret_cast<char*>(p.ws) +
                                            (parts * p.d * 2 + 255) / 256 * 256);
    }
    if (p.d == 64)
      launch_mfma<64>(dim3(p.workers), p, s);
    else
      launch_mfma<72>(dim3(p.workers), p, s);
    if (cut) {
      if (p.d == 64)
        hipLaunchKernelGGL(attn_merge_kernel<64>, dim3(MergeGeo<64>::BLOCKS, tiles),
                           dim3(MergeGeo<64>::THREADS), 0, s, p);
      else
        hipLaunchKernelGGL(attn_merge_kernel<72>, dim3(MergeGeo<72>::BLOCKS, tiles),
                           dim3(MergeGeo<72>::THREADS), 0, s, p);
    }
    return hipGetLastError();
  }
  if (dtype == kBF16) return launch_simt<bf16>(p, s);
  return launch_simt<float>(p, s);
}

}  // namespace orch
