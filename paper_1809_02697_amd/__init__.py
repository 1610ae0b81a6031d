"""Blocked-layout CNN inference on MI355X (gfx950).

The package holds the Python binding of the C-ABI library ``libneo`` (see
``paper_1809_02697_amd.neo``) and the seeded synthetic workloads
(``paper_1809_02697_amd.workloads``).  Importing the package imports neither,
so a caller that only needs the workloads never loads the HIP library.
"""
