"""SAEF (step-ahead error feedback) scaled-sign compression round on MI355X.

The compute path is the HIP library ``libsaef.so`` built from ``csrc/``; the
Python binding in ``saef`` only marshals arguments to its C entry points.
``workloads`` holds the seeded synthetic inputs.  Importing this package does
not load the library; importing ``paper_2008_05823_amd.saef`` does, and fails
loudly if it is missing.
"""
