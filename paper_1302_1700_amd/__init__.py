"""Fragment-based image scanning with deep max-pooling CNNs on MI355X (gfx950).

The scan lives in the HIP library ``libfragscan.so`` behind the C-ABI declared
in ``include/fragscan.h``; ``paper_1302_1700_amd.fragscan`` is its thin Python
binding.  ``paper_1302_1700_amd.workloads`` draws seeded nets and images.
"""
