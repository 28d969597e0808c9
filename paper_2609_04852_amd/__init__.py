"""MI355X-native KVMem decode-step path (arXiv 2609.04852).

Importing the package loads nothing: the HIP library is opened on first use by
`paper_2609_04852_amd.kvmem`, which raises if it has not been built.
"""
