// Entropy coding of the quantised latent (Fig. 4 "AE" / "AD", Fig. 6): rANS
// (Duda 2013, range variant: 32-bit state in [2^16, 2^32), 16-bit words,
// M = 2^16) on quantised-scale Gaussian tables.
//
// A stream is 8192 symbols coded by the 64 lanes of one wave in lock step:
// symbol i of the stream belongs to lane i % 64 at step i / 64.  At every
// (step, sub-symbol) the lanes that move a word do so in lane order (ballot +
// popcount give each its slot), so a stream is one contiguous run of words.
// An escaped symbol (|q| beyond its table) continues with one 16-bit field
// of frequency 1: 32768 * sign + |q| - R - 1.
//
// Every coder kernel first stages what its sequential loop touches into LDS
// with direct global->LDS loads issued back to back and one wait (the tables,
// the stream's symbols and scale indices, the decoder also the stream's
// words), so the loop over the 128 steps never waits on global memory.
//
// k_rans_encode  one wave per stream: encodes backwards into the stream's
//                scratch slot, words ending at the slot's end
// k_rans_frame   one workgroup: prefix sum of the stream lengths, container
//                header and length table
// k_rans_pack    one workgroup per stream: copies the words into the container
// k_rans_index   one workgroup: checks a container, prefix sum of its lengths
// k_rans_decode  one wave per stream: decodes forward, every word read bounded
//                by the stream's length; flags a truncated or inconsistent
//                stream instead of reading past it
#include "common.hpp"
#include "internal.hpp"

namespace nc {

namespace {

constexpr uint32_t kRansL = 1u << 16;

// Direct global->LDS load of 4 bytes per lane: lane l's bytes land at
// lds_wave_base + 4 l.  Callers wait with s_waitcnt vmcnt before reading.
__device__ __forceinline__ void dma4(const void* g, const void* lds_wave_base) {
  const uint32_t m = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)lds_wave_base;
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off" ::"v"(g), "s"(m) : "memory", "m0");
}

// Stages n16 16-byte chunks from g into LDS at lds (one wave).
__device__ __forceinline__ void stage16(const void* g, void* lds, int n16, int lane) {
  for (int i = 0; i < n16; i += 64)
    if (i + lane < n16) dma16((const uint8_t*)g + 16 * (i + lane), (uint8_t*)lds + 16 * i);
}

// x / f and x mod f for 1 <= f < 2^16 and x < f 2^16 (the quotient is below
// 2^16): the fp32 estimate x * rcp(f) is within 2^-6 of x / f (relative error
// at most about 2^-22 on a quotient below 2^16), so its truncation is off by
// at most one and a single correction each way makes it exact.
__device__ __forceinline__ uint32_t divmod16(uint32_t x, uint32_t f, uint32_t& r) {
  uint32_t qd = (uint32_t)((float)x * __builtin_amdgcn_rcpf((float)f));
  int32_t rr = (int32_t)(x - __umul24(qd, f));
  if (rr < 0) {
    --qd;
    rr += (int32_t)f;
  } else if (rr >= (int32_t)f) {
    ++qd;
    rr -= (int32_t)f;
  }
  r = (uint32_t)rr;
  return qd;
}

}  // namespace

// One wave (workgroup) per stream.  After staging, a parallel pass turns
// every symbol into its table entry (start << 16 | frequency); the sequential
// loop then reads one LDS word per step.
__global__ __launch_bounds__(64) void k_rans_encode(const int16_t* q, const uint8_t* kidx, int64_t n,
                                                  const uint16_t* tab, uint16_t* scratch, int64_t max_words,
                                                  uint32_t* lens) {
  __shared__ __align__(16) uint16_t st[kTabEncU16];
  __shared__ __align__(16) uint32_t scf[kRansStream];
  __shared__ __align__(16) int16_t sq[kRansStream];
  __shared__ __align__(16) uint8_t sk[kRansStream];
  const int lane = threadIdx.x;
  const int64_t s = blockIdx.x;
  const int64_t base = s * kRansStream;
  const int cnt = (int)min((int64_t)kRansStream, n - base);
  const int steps = (cnt + 63) / 64;
  stage16(tab, st, kTabEncU16 / 8, lane);
  const int nq = cnt / 8, nk = cnt / 16;  // whole 16-byte chunks; q and k are 16-byte aligned
  stage16(q + base, sq, nq, lane);
  stage16(kidx + base, sk, nk, lane);
  if (8 * nq + lane < cnt) sq[8 * nq + lane] = q[base + 8 * nq + lane];
  if (16 * nk + lane < cnt) sk[16 * nk + lane] = kidx[base + 16 * nk + lane];
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  // table entry of every symbol (positions past cnt get values that are never used)
  const uint16_t* sst = st + kTabStarts;
#pragma unroll 8
  for (int t = 0; t < steps; ++t) {
    const int li = t * 64 + lane;
    const int qv = sq[li];
    const int k = min((int)sk[li], kCoderScales - 1);
    const int R = st[k], o = st[kCoderScales + k];
    const int i = (qv < -R || qv > R) ? 2 * R + 1 : qv + R;
    const uint32_t c = sst[o + i], cn = sst[o + i + 1];
    scf[li] = (c << 16) | ((cn - c) & 0xFFFFu);
  }
  __syncthreads();
  uint16_t* end = scratch + (s + 1) * max_words;
  const uint64_t below = (1ull << lane) - 1;
  int p = 0;  // words written, counted back from the end
  uint32_t x = kRansL;
  for (int t = steps - 1; t >= 0; --t) {
    const int li = t * 64 + lane;
    const bool act = li < cnt;
    const uint32_t e = scf[li];
    const uint32_t c = e >> 16, f = act ? (e & 0xFFFFu) : 1u;
    const bool esc = act && c + f == 65536u;  // the last entry of a table is the escape
    if (__ballot(esc)) {
      // the field follows the escape in decoding order, so it is coded first;
      // with frequency 1 every escaped state moves a word out
      const uint64_t m = __ballot(esc);
      const int cw = (int)__popcll(m);  // __popcll is unsigned: keep the slot arithmetic signed
      if (esc) {
        const int qv = sq[li];
        const int R = st[min((int)sk[li], kCoderScales - 1)];
        const uint32_t fld = (qv < 0 ? 32768u : 0u) + (uint32_t)(abs(qv) - R - 1);
        end[(int)__popcll(m & below) - (p + cw)] = (uint16_t)(x & 0xFFFFu);
        x = (x & 0xFFFF0000u) | fld;
      }
      p += cw;
    }
    const bool emit = act && x >= (f << 16);
    const uint64_t m = __ballot(emit);
    const int cw = (int)__popcll(m);
    if (emit) {
      end[(int)__popcll(m & below) - (p + cw)] = (uint16_t)(x & 0xFFFFu);
      x >>= 16;
    }
    p += cw;
    if (act) {
      uint32_t r;
      const uint32_t qd = divmod16(x, f, r);
      x = (qd << 16) + r + c;
    }
  }
  // the 64 final states open the stream: lane l at words 2l (high) and 2l + 1
  end[-(p + 128) + 2 * lane] = (uint16_t)(x >> 16);
  end[-(p + 128) + 2 * lane + 1] = (uint16_t)(x & 0xFFFFu);
  p += 128;
  if (lane == 0) lens[s] = (uint32_t)p;
}

// Block-wide exclusive prefix sum of one value per thread (1024 threads).
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* total, uint32_t* sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t inc = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t o = __shfl_up(inc, off, 64);
    if (lane >= off) inc += o;
  }
  if (lane == 63) sh[wave] = inc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t acc = 0;
    for (int w = 0; w < 16; ++w) {
      const uint32_t t = sh[w];
      sh[w] = acc;
      acc += t;
    }
    sh[16] = acc;
  }
  __syncthreads();
  const uint32_t r = sh[wave] + inc - v;
  *total = sh[16];
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(1024) void k_rans_frame(const uint32_t* lens, int64_t n, uint32_t* offs, uint8_t* out,
                                                   uint64_t* nbytes) {
  __shared__ uint32_t sh[17];
  const int ns = (int)((n + kRansStream - 1) / kRansStream);
  uint16_t* ltab = (uint16_t*)(out + kRansHeader);
  uint32_t carry = 0;
  for (int b = 0; b < ns; b += 1024) {
    const int i = b + threadIdx.x;
    const uint32_t v = i < ns ? lens[i] : 0u;
    uint32_t tot;
    const uint32_t ex = block_excl_scan(v, &tot, sh);
    if (i < ns) {
      offs[i] = carry + ex;
      ltab[i] = (uint16_t)v;
    }
    carry += tot;
  }
  if (threadIdx.x == 0) {
    uint32_t* h = (uint32_t*)out;
    h[0] = kRansMagic;
    h[1] = kRansVersion;
    h[2] = (uint32_t)n;
    h[3] = (uint32_t)kRansStream;
    h[4] = (uint32_t)ns;
    if (ns & 1) ltab[ns] = 0;  // pad to 4 bytes
    *nbytes = (uint64_t)rans_payload_offset(ns) + 2ull * carry;
  }
}

__global__ __launch_bounds__(256) void k_rans_pack(const uint16_t* scratch, int64_t max_words, const uint32_t* lens,
                                                 const uint32_t* offs, int64_t n, uint8_t* out) {
  const int ns = (int)((n + kRansStream - 1) / kRansStream);
  const int s = blockIdx.x;
  if (s >= ns) return;
  const uint32_t len = lens[s];
  const uint16_t* src = scratch + (int64_t)(s + 1) * max_words - len;
  uint16_t* dst = (uint16_t*)(out + rans_payload_offset(ns)) + offs[s];
  for (uint32_t i = threadIdx.x; i < len; i += 256) dst[i] = src[i];
}

__global__ __launch_bounds__(1024) void k_rans_index(const uint8_t* in, uint64_t in_bytes, int64_t n, uint32_t* offs,
                                                   uint32_t* lens, int32_t* status) {
  __shared__ uint32_t sh[17];
  __shared__ int bad;
  const int ns = (int)((n + kRansStream - 1) / kRansStream);
  if (threadIdx.x == 0) {
    bad = 0;
    if (in_bytes < (uint64_t)rans_payload_offset(ns)) {
      bad = 1;
    } else {
      const uint32_t* h = (const uint32_t*)in;
      bad = !(h[0] == kRansMagic && h[1] == kRansVersion && h[2] == (uint32_t)n && h[3] == (uint32_t)kRansStream &&
              h[4] == (uint32_t)ns);
    }
  }
  __syncthreads();
  const bool ok = !bad;
  const uint16_t* ltab = (const uint16_t*)(in + kRansHeader);
  uint32_t carry = 0;
  for (int b = 0; b < ns; b += 1024) {
    const int i = b + threadIdx.x;
    const uint32_t v = (ok && i < ns) ? ltab[i] : 0u;
    uint32_t tot;
    const uint32_t ex = block_excl_scan(v, &tot, sh);
    if (i < ns) {
      offs[i] = carry + ex;
      lens[i] = v;
    }
    carry += tot;
  }
  if (threadIdx.x == 0) {
    int st = bad ? 1 : 0;
    if (!bad && (uint64_t)rans_payload_offset(ns) + 2ull * carry > in_bytes) st = 1;
    status[0] = st;
    status[1] = 0;
  }
}

// One wave (workgroup) per stream.  LDS holds the whole coder table block,
// the stream's scale indices and the stream's words (word i at sw[par + i],
// par the parity of the stream's start, so that whole dwords can be staged).
__global__ __launch_bounds__(64) void k_rans_decode(const uint8_t* in, const uint8_t* kidx, int64_t n,
                                                  const uint16_t* tab, const uint32_t* offs, const uint32_t* lens,
                                                  int16_t* q, int32_t* status) {
  __shared__ __align__(16) uint16_t st[kTabU16];
  __shared__ __align__(16) uint8_t sk[kRansStream];
  __shared__ __align__(16) uint16_t sw[kRansMaxWords + 2];
  const int lane = threadIdx.x;
  const int64_t s = blockIdx.x;
  const int ns = (int)((n + kRansStream - 1) / kRansStream);
  const int64_t base = s * kRansStream;
  const int cnt = (int)min((int64_t)kRansStream, n - base);
  const int steps = (cnt + 63) / 64;
  const bool head_ok = status[0] == 0;  // status[0]: container check, status[1]: stream errors
  int err = 0;
  uint32_t len = head_ok ? lens[s] : 0u;
  if (len > (uint32_t)kRansMaxWords) {
    err |= 2;
    len = 0;
  }
  if (len < 128) err |= 2;
  // the stream's words are u16 indices [g0, g1) of the container
  const uint64_t g0 = (uint64_t)(rans_payload_offset(ns) / 2) + (head_ok ? offs[s] : 0u), g1 = g0 + len;
  const int par = (int)(g0 & 1);
  stage16(tab, st, kTabU16 / 8, lane);
  const int nk = cnt / 16;  // k is 16-byte aligned
  stage16(kidx + base, sk, nk, lane);
  if (16 * nk + lane < cnt) sk[16 * nk + lane] = kidx[base + 16 * nk + lane];
  {
    // whole dwords d0 .. d1 - 1 inside [g0, g1); dword d lands at sw[2 (d - g0 / 2)]
    const uint64_t d0 = (g0 + 1) / 2, d1 = g1 / 2;
    const int nd = d1 > d0 ? (int)(d1 - d0) : 0;
    const uint32_t* src = (const uint32_t*)in + d0;
    uint16_t* dst = sw + 2 * (d0 - g0 / 2);
    for (int i = 0; i < nd; i += 64)
      if (i + lane < nd) dma4(src + i + lane, dst + 2 * i);
    const uint16_t* in16 = (const uint16_t*)in;
    if (lane == 0 && len > 0 && par) sw[1] = in16[g0];                          // odd first word
    if (lane == 1 && len > 0 && (g1 & 1)) sw[par + len - 1] = in16[g1 - 1];   // odd last word
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  const uint16_t* sst = st + kTabStarts;
  const uint16_t* sbk = st + kTabBuckets;
  const uint64_t below = (1ull << lane) - 1;
  auto word = [&](uint32_t i) -> uint32_t { return i < len ? (uint32_t)sw[par + i] : 0u; };
  uint32_t x = (word(2 * lane) << 16) | word(2 * lane + 1);
  uint32_t pos = 128;
  // lane-ordered renormalisation reads of the lanes in need
  auto refill = [&](bool need) {
    const uint64_t m = __ballot(need);
    if (need) {
      const uint32_t i = pos + (uint32_t)__popcll(m & below);
      if (i >= len) err |= 2;
      x = (x << 16) | word(i);
    }
    pos += (uint32_t)__popcll(m);
  };
  for (int t = 0; t < steps; ++t) {
    const int li = t * 64 + lane;
    const bool act = li < cnt;
    // positions past cnt read values that are never used; every index stays inside the tables
    const int k = min((int)sk[li], kCoderScales - 1);
    const int R = st[k], o = st[kCoderScales + k];
    const uint32_t slot = x & 0xFFFFu;
    // the bucket bounds the entry holding the slot; a binary search finds it
    int lo = sbk[k * 257 + (slot >> 8)], hi = sbk[k * 257 + (slot >> 8) + 1];
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (sst[o + mid] <= slot) lo = mid;
      else hi = mid - 1;
    }
    const uint32_t c = sst[o + lo], f = ((uint32_t)sst[o + lo + 1] - c) & 0xFFFFu;
    const bool esc = act && lo == 2 * R + 1;
    if (act) x = f * (x >> 16) + slot - c;
    refill(act && x < kRansL);
    int qv = lo - R;
    if (__ballot(esc)) {
      const uint32_t fld = x & 0xFFFFu;
      if (esc) x >>= 16;
      refill(esc);
      if (esc) {
        const int mag = R + 1 + (int)(fld & 32767u);
        qv = (fld >> 15) ? -mag : mag;
      }
    }
    if (act) q[base + li] = (int16_t)max(min(qv, 32767), -32768);
  }
  if (head_ok && (x != kRansL || pos != len)) err |= 4;
  if (err) atomicOr(status + 1, err);
}

__global__ void k_rans_status(const int32_t* status, int32_t* out) { *out = status[0] | status[1]; }

hipError_t launch_rans_encode(const int16_t* q, const uint8_t* k, int64_t n, const uint16_t* tab, uint16_t* scratch,
                              int64_t max_words, uint32_t* lens, uint32_t* offs, uint8_t* out, uint64_t* nbytes,
                              hipStream_t st) {
  const int64_t ns = (n + kRansStream - 1) / kRansStream;
  if (ns <= 0 || ns > 65535) return hipErrorInvalidValue;
  launch(k_rans_encode, dim3((unsigned)ns), dim3(64), st, q, k, n, tab, scratch, max_words, lens);
  launch(k_rans_frame, dim3(1), dim3(1024), st, (const uint32_t*)lens, n, offs, out, nbytes);
  launch(k_rans_pack, dim3((unsigned)ns), dim3(256), st, (const uint16_t*)scratch, max_words, (const uint32_t*)lens,
         (const uint32_t*)offs, n, out);
  return hipGetLastError();
}

hipError_t launch_rans_decode(const uint8_t* in, uint64_t in_bytes, const uint8_t* k, int64_t n, const uint16_t* tab,
                              uint32_t* offs, uint32_t* lens, int16_t* q, int32_t* status, int32_t* status_out,
                              hipStream_t st) {
  const int64_t ns = (n + kRansStream - 1) / kRansStream;
  if (ns <= 0 || ns > 65535) return hipErrorInvalidValue;
  launch(k_rans_index, dim3(1), dim3(1024), st, in, in_bytes, n, offs, lens, status);
  launch(k_rans_decode, dim3((unsigned)ns), dim3(64), st, in, k, n, tab, (const uint32_t*)offs, (const uint32_t*)lens,
         q, status);
  if (status_out) launch(k_rans_status, dim3(1), dim3(1), st, (const int32_t*)status, status_out);
  return hipGetLastError();
}

}  // namespace nc
