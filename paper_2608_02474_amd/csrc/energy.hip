// Audio energy anchor (Sec. 3.3, "Cross-modal Saliency Anchors"): per-segment
// STFT power, pooled into mel-width bands and latent frames.
//
// Kernel 1 (energy_frames): one workgroup per (segment, STFT frame), in fp64.
// For a power-of-two n_fft, an in-place radix-2 FFT in LDS (log2 n_fft
// barrier-separated butterfly stages); for any other even n_fft, each thread
// evaluates whole one-sided bins k directly from the DFT sum over a
// full-period twiddle table.  |X_k|^2 and each bin's band go to LDS, and one
// wave per band sums its bins.  Both stay within fp64 rounding of the
// definition.
// Kernel 2 (energy_reduce): one workgroup sums the per-frame band energies of
// each (segment, band) in frame order (one thread each), then each segment's
// bands, and forms e_t and e_t / max e.
#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace echo {

constexpr int kEnergyThreads = 256;   // energy_reduce (power of two: tree reduction)
constexpr int kFrameThreads = 512;    // energy_frames: one thread per one-sided bin up to n_fft 1022
constexpr int kFftThreads = 256;     // energy_frames_fft
constexpr int kMaxFft = 2048;

__device__ __forceinline__ int band_of_bin(int k, int n_fft, int sr, int n_bands) {
  const double mel_top = 2595.0 * log10(1.0 + (0.5 * sr) / 700.0);
  const double width = mel_top / n_bands;
  const double f = static_cast<double>(k) * sr / n_fft;
  const double m = 2595.0 * log10(1.0 + f / 700.0);
  int b = static_cast<int>(floor(m / width));
  return b < n_bands - 1 ? b : n_bands - 1;
}

// Per-band sums of the bin powers, one wave per band (lanes take bins
// lane, lane + 64, ...; fp64 throughout).
__device__ __forceinline__ void band_sums(const double* pw, const int* bandof, int nbins, int n_bands,
                                          double* __restrict__ out) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave, nw = blockDim.x / kWave;
  for (int band = wave; band < n_bands; band += nw) {
    double acc = 0.0;
    for (int k = lane; k < nbins; k += kWave)
      if (bandof[k] == band) acc += pw[k];
    acc = wave_sum(acc);
    if (lane == 0) out[band] = acc;
  }
}

// Radix-2 path for a power-of-two n_fft: one workgroup of kFftThreads per
// (segment, frame).  The windowed frame is placed in bit-reversed order and
// transformed in place by log2(n_fft) decimation-in-time butterfly stages in
// fp64 (twiddles exp(-2 pi i j / n_fft) from an LDS table); then the one-sided
// powers and the band sums as in the direct path.
__global__ void __launch_bounds__(kFftThreads)
energy_frames_fft(const float* __restrict__ audio, int64_t n_samples, int T, int n_fft, int log2n, int hop,
                  int n_bands, int sr, int max_frames, double* __restrict__ part) {
  extern __shared__ double lds[];
  double* re = lds;                       // [n_fft]
  double* im = lds + n_fft;               // [n_fft]
  double* twc = lds + 2 * n_fft;          // [n_fft/2] cos(2 pi j / n_fft)
  double* tws = twc + n_fft / 2;          // [n_fft/2] -sin(2 pi j / n_fft)
  double* pw = tws + n_fft / 2;           // [n_fft/2 + 1]
  int* bandof = reinterpret_cast<int*>(pw + n_fft / 2 + 1);  // [n_fft/2 + 1]
  const int t = blockIdx.y, f = blockIdx.x;
  const int64_t a = (static_cast<int64_t>(t) * n_samples) / T;
  const int64_t b = (static_cast<int64_t>(t + 1) * n_samples) / T;
  const int64_t len = b - a;
  const int nf = len < n_fft ? 1 : static_cast<int>(1 + (len - n_fft) / hop);
  double* out = part + (static_cast<int64_t>(t) * max_frames + f) * n_bands;
  if (f >= nf) {
    for (int i = threadIdx.x; i < n_bands; i += blockDim.x) out[i] = 0.0;
    return;
  }
  const int64_t start = a + static_cast<int64_t>(f) * hop;
  for (int n = threadIdx.x; n < n_fft; n += blockDim.x) {
    const double w = 0.5 - 0.5 * cospi(2.0 * n / n_fft);  // periodic Hann
    const int64_t sidx = start + n;
    const double v = (sidx < b) ? static_cast<double>(audio[sidx]) : 0.0;
    const int r = static_cast<int>(__brev(static_cast<unsigned>(n)) >> (32 - log2n));
    re[r] = w * v;
    im[r] = 0.0;
  }
  for (int j = threadIdx.x; j < n_fft / 2; j += blockDim.x) {
    double sn, cs;
    sincospi(2.0 * j / n_fft, &sn, &cs);
    twc[j] = cs;
    tws[j] = -sn;
  }
  __syncthreads();
  for (int st = 1; st <= log2n; ++st) {
    const int half = 1 << (st - 1);
    for (int bf = threadIdx.x; bf < n_fft / 2; bf += blockDim.x) {
      const int pos = bf & (half - 1);
      const int i0 = ((bf >> (st - 1)) << st) + pos, i1 = i0 + half;
      const int tw = pos << (log2n - st);
      const double wr = twc[tw], wi = tws[tw];
      const double br = re[i1], bi = im[i1];
      const double xr = br * wr - bi * wi, xi = br * wi + bi * wr;
      const double ar = re[i0], ai = im[i0];
      re[i0] = ar + xr;
      im[i0] = ai + xi;
      re[i1] = ar - xr;
      im[i1] = ai - xi;
    }
    __syncthreads();
  }
  const int nbins = n_fft / 2 + 1;
  for (int k = threadIdx.x; k < nbins; k += blockDim.x) {
    pw[k] = re[k] * re[k] + im[k] * im[k];
    bandof[k] = band_of_bin(k, n_fft, sr, n_bands);
  }
  __syncthreads();
  band_sums(pw, bandof, nbins, n_bands, out);
}

__global__ void __launch_bounds__(kFrameThreads)
energy_frames(const float* __restrict__ audio, int64_t n_samples, int T, int n_fft, int hop,
              int n_bands, int sr, int max_frames, double* __restrict__ part) {
  extern __shared__ double lds[];
  double* xw = lds;                 // [n_fft] windowed frame
  double* tc = lds + n_fft;         // [n_fft] cos(2 pi m / n_fft)
  double* ts = lds + 2 * n_fft;     // [n_fft] sin(2 pi m / n_fft)
  double* pw = lds + 3 * n_fft;     // [n_fft/2 + 1] |X_k|^2
  int* bandof = reinterpret_cast<int*>(lds + 3 * n_fft + n_fft / 2 + 1);  // [n_fft/2 + 1] band of bin k
  const int t = blockIdx.y, f = blockIdx.x;
  const int64_t a = (static_cast<int64_t>(t) * n_samples) / T;
  const int64_t b = (static_cast<int64_t>(t + 1) * n_samples) / T;
  const int64_t len = b - a;
  const int nf = len < n_fft ? 1 : static_cast<int>(1 + (len - n_fft) / hop);
  double* out = part + (static_cast<int64_t>(t) * max_frames + f) * n_bands;
  if (f >= nf) {  // frame slot past this segment's frame count: contributes zero
    for (int i = threadIdx.x; i < n_bands; i += blockDim.x) out[i] = 0.0;
    return;
  }
  const int64_t start = a + static_cast<int64_t>(f) * hop;
  for (int n = threadIdx.x; n < n_fft; n += blockDim.x) {
    const double w = 0.5 - 0.5 * cospi(2.0 * n / n_fft);      // periodic Hann
    const int64_t s = start + n;
    const double v = (s < b) ? static_cast<double>(audio[s]) : 0.0;  // zero-pad short segments
    xw[n] = w * v;
    double sn, cs;
    sincospi(2.0 * n / n_fft, &sn, &cs);
    tc[n] = cs;
    ts[n] = sn;
  }
  __syncthreads();
  const int nbins = n_fft / 2 + 1;
  for (int k = threadIdx.x; k < nbins; k += blockDim.x) {
    // four independent partial sums over n = 4j + u, so that four twiddle
    // reads and FMA chains are in flight at once (an even n_fft that is not
    // a multiple of 4 leaves two terms for the tail)
    double re[4] = {0.0, 0.0, 0.0, 0.0}, im[4] = {0.0, 0.0, 0.0, 0.0};
    int m[4];  // (k * n) mod n_fft for the four current n, advanced by 4k
#pragma unroll
    for (int u = 0; u < 4; ++u) m[u] = (k * u) % n_fft;
    const int step = (4 * k) % n_fft;
    int n = 0;
    for (; n + 4 <= n_fft; n += 4) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const double x = xw[n + u];
        re[u] = fma(x, tc[m[u]], re[u]);
        im[u] = fma(-x, ts[m[u]], im[u]);
        m[u] += step;
        if (m[u] >= n_fft) m[u] -= n_fft;
      }
    }
    for (int u = 0; n + u < n_fft; ++u) {
      const double x = xw[n + u];
      re[u] = fma(x, tc[m[u]], re[u]);
      im[u] = fma(-x, ts[m[u]], im[u]);
    }
    const double r = (re[0] + re[1]) + (re[2] + re[3]);
    const double i = (im[0] + im[1]) + (im[2] + im[3]);
    pw[k] = r * r + i * i;
    bandof[k] = band_of_bin(k, n_fft, sr, n_bands);
  }
  __syncthreads();
  band_sums(pw, bandof, nbins, n_bands, out);
}

__global__ void __launch_bounds__(kEnergyThreads)
energy_reduce(const double* __restrict__ part, int T, int max_frames, int n_bands,
              float* __restrict__ band_energy, float* __restrict__ frame_energy,
              float* __restrict__ frame_weight, double* __restrict__ e_scratch) {
  __shared__ double red[kEnergyThreads];
  // (1) one thread per (segment, band): the band's frames summed in frame
  //     order; the fp64 band sums go to e_scratch[T + t * n_bands + band]
  double* bsum = e_scratch + T;
  for (int i = threadIdx.x; i < T * n_bands; i += blockDim.x) {
    const int t = i / n_bands, band = i % n_bands;
    const double* src = part + static_cast<int64_t>(t) * max_frames * n_bands + band;
    double acc = 0.0;
    // unrolled so that eight frames' loads are in flight; the additions keep
    // frame order
#pragma unroll 8
    for (int f = 0; f < max_frames; ++f) acc += src[static_cast<int64_t>(f) * n_bands];
    bsum[i] = acc;
    band_energy[i] = static_cast<float>(acc);
  }
  __syncthreads();
  // (2) one thread per segment: its bands in band order
  double local_max = 0.0;
  for (int t = threadIdx.x; t < T; t += blockDim.x) {
    double tot = 0.0;
    for (int band = 0; band < n_bands; ++band) tot += bsum[t * n_bands + band];
    const double e = sqrt(tot);
    e_scratch[t] = e;
    frame_energy[t] = static_cast<float>(e);
    local_max = fmax(local_max, e);
  }
  red[threadIdx.x] = local_max;
  __syncthreads();
  for (int s = blockDim.x / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) red[threadIdx.x] = fmax(red[threadIdx.x], red[threadIdx.x + s]);
    __syncthreads();
  }
  const double mx = red[0];
  for (int t = threadIdx.x; t < T; t += blockDim.x)
    frame_weight[t] = mx > 0.0 ? static_cast<float>(e_scratch[t] / mx) : 1.0f;
}

int energy_max_frames(int64_t n_samples, int T, int n_fft, int hop) {
  // the longest segment has ceil(n / T) samples
  const int64_t longest = (n_samples + T - 1) / T;
  return longest < n_fft ? 1 : static_cast<int>(1 + (longest - n_fft) / hop);
}

hipError_t launch_energy(const float* audio, int64_t n_samples, int T, int sr, int n_fft, int hop,
                         int n_bands, float* band_energy, float* frame_energy, float* frame_weight,
                         double* part, double* e_scratch, hipStream_t stream) {
  const int mf = energy_max_frames(n_samples, T, n_fft, hop);
  hipError_t e;
  if ((n_fft & (n_fft - 1)) == 0) {
    int log2n = 0;
    while ((1 << log2n) < n_fft) ++log2n;
    const size_t lds = sizeof(double) * (3 * n_fft + n_fft / 2 + 1) + sizeof(int) * (n_fft / 2 + 1);
    e = ECHO_LAUNCH("energy_frames", energy_frames_fft, dim3(mf, T), dim3(kFftThreads), lds, stream, audio,
                    n_samples, T, n_fft, log2n, hop, n_bands, sr, mf, part);
  } else {
    const size_t lds = sizeof(double) * (3 * n_fft + n_fft / 2 + 1) + sizeof(int) * (n_fft / 2 + 1);
    e = ECHO_LAUNCH("energy_frames", energy_frames, dim3(mf, T), dim3(kFrameThreads), lds, stream, audio,
                    n_samples, T, n_fft, hop, n_bands, sr, mf, part);
  }
  if (e != hipSuccess) return e;
  return ECHO_LAUNCH("energy_reduce", energy_reduce, dim3(1), dim3(kEnergyThreads), 0, stream, part, T,
                     mf, n_bands, band_energy, frame_energy, frame_weight, e_scratch);
}

}  // namespace echo
