/*
 * kred_probe: sustained-rate microbenchmarks of one gfx950 device, for the
 * measured side of a roofline next to MI355X's published peaks.  Separate from
 * the reduction library (libkred_probe.so); bench.py reports its figures.
 */
#ifndef KRED_PROBE_H
#define KRED_PROBE_H

#ifdef __cplusplus
extern "C" {
#endif

typedef struct kred_peak {
  double fma_tflops;  /* sustained fp32 FMA rate, 2 flops per FMA: non-packed v_fma with every
                         operand in VGPRs, 16 independent chains per lane, 8 waves per SIMD */
  double exp_gops;    /* sustained v_exp_f32 rate, in 10^9 per second, same occupancy */
  double sclk_mhz;    /* shader clock during the FMA probe: s_memtime against s_memrealtime
                         (a constant 100 MHz) in one wave */
  double fma_ms;      /* duration of the timed FMA launch (HIP events) */
  double exp_ms;      /* duration of the timed exp launch */
  int cus;            /* compute units of the device */
} kred_peak;

/*
 * Run the probes on HIP device `device` (about 50 ms; allocates and frees a
 * few MB, synchronises, restores the caller's current device).  Fills *res.
 * Returns 0 on success, non-zero on a HIP failure (res then partly filled).
 */
int kred_probe_peak(int device, kred_peak* res);

#ifdef __cplusplus
}
#endif

#endif /* KRED_PROBE_H */
