"""OptCC schedule execution on one MI355X (gfx950).

The library (``liboptcc.so``, C ABI in ``include/optcc.h``) plans the OptCC
AllReduce schedule for a bandwidth profile, evaluates its closed-form time and
lower bound, and executes every step of the schedule with HIP kernels over p
rank buffers held in one GPU's HBM.  ``paper_2606_01680_amd.optcc`` is the
ctypes binding; ``workloads`` draws seeded synthetic inputs.
"""
