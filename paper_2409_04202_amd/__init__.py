"""MI355X (gfx950) executor for AllReduce plans of GenModel / GenTree
(arXiv 2409.04202): n emulated processors whose buffers live in one GPU.

* ``paper_2409_04202_amd.arplan``    -- ctypes binding of the C-ABI library
  (``include/ar_plan.h``); importing it loads the HIP library and raises if it
  has not been built.
* ``paper_2409_04202_amd.workloads`` -- seeded synthetic workloads.
* ``paper_2409_04202_amd.build``     -- compiles the library with hipcc.
"""
