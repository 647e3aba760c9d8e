"""MI355X-native PD scan (Flash PD-SSM's recurrence h_t = P_{k_t} D_t h_{t-1} + b_t,
y_t = Re<c_t, h_t>) as hand-written HIP kernels for gfx950 behind a C ABI.

``paper_2605_19150_amd.pdssm`` is the thin ctypes binding over ``libpdssm.so``;
``paper_2605_19150_amd.inputs`` draws seeded synthetic inputs.  Importing the
package loads nothing; the binding loads the library on first use and raises if
it is missing.
"""
