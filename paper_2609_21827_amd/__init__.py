"""RheoSampling hot path on AMD Instinct MI355X (gfx950).

The product is the C-ABI library ``librheo.so`` (include/rheo.h) built from
``csrc/`` by ``build.py``; ``binding`` wraps it for Python (torch buffers and
streams) and ``driver`` runs whole decoding steps over a draft / target model
callback.  Importing the package does not load the library; importing
``binding`` does, and fails loudly when it has not been built.
"""
