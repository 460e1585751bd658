"""MI355X-native verifier scoring pass of VideoSpeculateRAG (arxiv 2601.01513).

The scoring pass lives in a HIP library (``libvsr.so``, C ABI declared in
``include/vsr.h``); ``binding`` marshals arguments to it. ``workload`` holds
the seeded synthetic inputs.
"""
