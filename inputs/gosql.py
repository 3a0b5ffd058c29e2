"""A Go-like language with embedded SQL: grammar, documents and vocabulary.

Stand-in for the paper's programming-language workloads at their scale
(Java, Go and SQL from The Stack, Sec. 4.1; their preprocessing cost,
Tab. preprocess), whose grammars and data are not available here.  The
grammar is our own and is LALR(1) as written:

* Go-like declarations and statements: package/import, func and method
  declarations, var/const/type declarations with struct and interface
  types, if/else, for (three-clause, condition, range), switch with case
  clauses, select, go/defer/return/goto/break/continue/fallthrough,
  assignments, short variable declarations, sends, increments;
* Go-like expressions: five binary precedence levels, unary operators and
  receive, selectors, indexing, slicing, type assertions, calls with
  variadic arguments, function literals, and composite literals of slice,
  array and map types (a named type followed by "{" would make headers
  like `if x {` ambiguous, so literals of named types are not part of it);
* an embedded SQL dialect, `sql(...)`: SELECT with joins, grouping, window
  functions, set operations and common table expressions; INSERT with
  ON CONFLICT, UPDATE, DELETE, CREATE TABLE/INDEX/VIEW, DROP, ALTER and
  transaction statements; SQL expressions with their own eight precedence
  levels, CASE, CAST, EXISTS and IN subqueries.

Statements end at a newline (the byte 0x0A, a terminal); other white space
and comments are ignored.  SQL keywords are upper case, Go's lower case.
"""
from __future__ import annotations

import functools

import numpy as np

from .grammar import Grammar, GrammarTables
from .vocab import Vocab, piece_vocab

GO_KEYWORDS = ["break", "case", "chan", "const", "continue", "default", "defer", "else", "fallthrough", "for",
               "func", "go", "goto", "if", "import", "interface", "map", "package", "range", "return", "select",
               "struct", "switch", "type", "var", "nil", "true", "false", "sql", "make", "new"]
GO_OPS = ["+", "-", "*", "/", "%", "&", "|", "^", "<<", ">>", "&^", "+=", "-=", "*=", "/=", "%=", "&=", "|=",
          "^=", "<<=", ">>=", "&^=", "&&", "||", "<-", "++", "--", "==", "<", ">", "=", "!", "!=", "<=", ">=",
          ":=", "...", "(", ")", "[", "]", "{", "}", ",", ";", ".", ":", "~"]
SQL_KEYWORDS = [
    "SELECT", "FROM", "WHERE", "GROUP", "BY", "HAVING", "ORDER", "ASC", "DESC", "NULLS", "FIRST", "LAST", "LIMIT",
    "OFFSET", "DISTINCT", "ALL", "AS", "JOIN", "INNER", "LEFT", "RIGHT", "FULL", "OUTER", "CROSS", "NATURAL", "ON",
    "USING", "UNION", "INTERSECT", "EXCEPT", "WITH", "RECURSIVE", "INSERT", "INTO", "VALUES", "DEFAULT", "UPDATE",
    "SET", "DELETE", "RETURNING", "CONFLICT", "DO", "NOTHING", "CREATE", "TABLE", "TEMPORARY", "IF", "NOT",
    "EXISTS", "PRIMARY", "KEY", "FOREIGN", "REFERENCES", "UNIQUE", "CHECK", "CONSTRAINT", "INDEX", "VIEW", "DROP",
    "ALTER", "ADD", "COLUMN", "RENAME", "TO", "CASCADE", "RESTRICT", "AND", "OR", "IS", "NULL", "LIKE", "ILIKE",
    "BETWEEN", "IN", "CASE", "WHEN", "THEN", "ELSE", "END", "CAST", "TRUE", "FALSE", "COUNT", "SUM", "AVG", "MIN",
    "MAX", "COALESCE", "NULLIF", "OVER", "PARTITION", "ROWS", "RANGE", "UNBOUNDED", "PRECEDING", "FOLLOWING",
    "CURRENT", "ROW", "FILTER", "INTEGER", "BIGINT", "SMALLINT", "TEXT", "VARCHAR", "CHAR", "BOOLEAN", "REAL",
    "DOUBLE", "PRECISION", "NUMERIC", "DECIMAL", "DATE", "TIME", "TIMESTAMP", "INTERVAL", "BLOB", "SERIAL",
    "EXTRACT", "BEGIN", "COMMIT", "ROLLBACK", "TRANSACTION", "LATERAL", "FETCH", "NEXT", "ONLY", "ANY", "SOME",
    "ROLLUP", "CUBE", "GROUPING", "SETS", "WINDOW", "MERGE", "MATCHED", "GRANT", "REVOKE", "PRIVILEGES", "PUBLIC",
    "TRIGGER", "BEFORE", "AFTER", "EACH", "FUNCTION", "EXECUTE", "EXPLAIN", "ANALYZE", "ARRAY", "OF",
    "SUBSTRING", "POSITION", "TRIM", "BOTH", "LEADING", "TRAILING", "OVERLAY", "PLACING", "FOR", "DISTINCT",
    "ESCAPE", "SIMILAR", "COPY", "FORMAT", "HEADER", "DELIMITER", "CSV", "SHOW", "RESET", "PREPARE",
    "DEALLOCATE", "TRUNCATE", "SCHEMA", "SEQUENCE", "INCREMENT", "START", "CURRENT_DATE", "CURRENT_TIME",
    "CURRENT_TIMESTAMP", "STDIN", "STDOUT", "RETURNS", "LANGUAGE", "WITHIN", "AT", "ZONE", "IMMUTABLE",
    "STABLE", "VOLATILE", "SETOF", "SKIP", "LOCKED", "NOWAIT", "SHARE", "MATERIALIZED", "REFRESH", "TYPE",
    "DATA", "ENUM", "COMMENT", "VACUUM", "NO"]
SQL_OPS = ["<>", "||", "->", "->>", "@>", "<@", "::"]


def gosql_grammar() -> GrammarTables:
    g = Grammar("file")
    g.regex("IDENT", r"[A-Za-z_][A-Za-z0-9_]*")
    g.regex("INT", r"[0-9]+|0[xX][0-9a-fA-F]+")
    g.regex("FLOAT", r"[0-9]+\.[0-9]+([eE][+-]?[0-9]+)?")
    g.regex("STRING", r'"([^"\\\n]|\\.)*"')
    g.regex("RAWSTRING", r"`[^`]*`")
    g.regex("SQ", r"'([^'\\\n]|\\.)*'")
    g.regex("PARAM", r"\$[0-9]+|\?")
    g.ignore("WS", r"[ \t\r]+")
    g.ignore("COMMENT", r"//[^\n]*")
    for k in GO_KEYWORDS + SQL_KEYWORDS:
        g.literal(k)
    for op in GO_OPS + SQL_OPS:
        g.literal(op)
    NL = g.literal("\n")
    L = lambda *xs: list(xs)
    q = lambda t: f'"{t}"'

    # ------------------------------------------------------------ file level
    g.rule("file", L(q("package"), "IDENT", NL, "top_items"))
    g.rule("top_items", [], L("top_items", "top_item"))
    g.rule("top_item", [NL], L("import_decl", NL), L("func_decl", NL), L("method_decl", NL), L("decl", NL))
    g.rule("import_decl", L(q("import"), "import_spec"), L(q("import"), q("("), "nl_lines", "import_lines", q(")")))
    g.rule("import_lines", [], L("import_lines", "import_spec", "nl_plus"))
    g.rule("import_spec", ["STRING"], L("IDENT", "STRING"), L(q("."), "STRING"))
    g.rule("nl_lines", [], L("nl_lines", NL))
    g.rule("nl_plus", [NL], L("nl_plus", NL))
    g.rule("func_decl", L(q("func"), "IDENT", "tparams_opt", "signature"),
           L(q("func"), "IDENT", "tparams_opt", "signature", "block"))
    g.rule("tparams_opt", [], L(q("["), "tparam_list", q("]")))
    g.rule("tparam_list", ["tparam"], L("tparam_list", q(","), "tparam"))
    g.rule("tparam", L("IDENT", "constraint"))
    g.rule("constraint", ["constraint_term"], L("constraint", q("|"), "constraint_term"))
    g.rule("constraint_term", ["type"], L(q("~"), "type"))
    g.rule("method_decl", L(q("func"), "receiver", "IDENT", "signature", "block"))
    g.rule("receiver", L(q("("), "IDENT", "recv_type", q(")")))
    g.rule("recv_type", ["IDENT"], L(q("*"), "IDENT"))
    g.rule("decl", ["var_decl"], ["const_decl"], ["type_decl"])
    g.rule("var_decl", L(q("var"), "var_spec"), L(q("var"), q("("), "nl_lines", "var_lines", q(")")))
    g.rule("var_lines", [], L("var_lines", "var_spec", "nl_plus"))
    g.rule("var_spec", L("ident_list", "type"), L("ident_list", "type", q("="), "expr_list"),
           L("ident_list", q("="), "expr_list"))
    g.rule("const_decl", L(q("const"), "const_spec"), L(q("const"), q("("), "nl_lines", "const_lines", q(")")))
    g.rule("const_lines", [], L("const_lines", "const_spec", "nl_plus"))
    g.rule("const_spec", L("ident_list", q("="), "expr_list"), L("ident_list", "type", q("="), "expr_list"),
           ["IDENT"])
    g.rule("type_decl", L(q("type"), "type_spec"), L(q("type"), q("("), "nl_lines", "type_lines", q(")")))
    g.rule("type_lines", [], L("type_lines", "type_spec", "nl_plus"))
    g.rule("type_spec", L("IDENT", "type"), L("IDENT", q("="), "type"))
    g.rule("ident_list", ["IDENT"], L("ident_list", q(","), "IDENT"))

    # ------------------------------------------------------------ types
    g.rule("type", ["type_name"], ["type_lit"])
    g.rule("type_name", ["IDENT"], L("IDENT", q("."), "IDENT"))
    g.rule("type_lit", ["pointer_type"], ["func_type"], ["interface_type"], ["chan_type"], ["literal_type"])
    g.rule("literal_type", ["slice_type"], ["array_type"], ["map_type"], ["struct_type"])
    g.rule("pointer_type", L(q("*"), "type"))
    g.rule("slice_type", L(q("["), q("]"), "type"))
    g.rule("array_type", L(q("["), "expr", q("]"), "type"), L(q("["), q("..."), q("]"), "type"))
    g.rule("map_type", L(q("map"), q("["), "type", q("]"), "type"))
    g.rule("chan_type", L(q("chan"), "type"))
    g.rule("func_type", L(q("func"), "signature"))
    g.rule("signature", ["params"], L("params", "result"))
    g.rule("result", ["type"], L(q("("), "type_list", q(")")))
    g.rule("type_list", ["type"], L("type_list", q(","), "type"))
    g.rule("params", L(q("("), q(")")), L(q("("), "param_list", q(")")), L(q("("), "param_list", q(","), q(")")))
    g.rule("param_list", ["param"], L("param_list", q(","), "param"))
    g.rule("param", L("IDENT", "type"), L("IDENT", q("..."), "type"))
    g.rule("struct_type", L(q("struct"), q("{"), q("}")), L(q("struct"), q("{"), NL, "field_lines", q("}")),
           L(q("struct"), q("{"), "inline_fields", q("}")))
    g.rule("inline_fields", ["field_decl"], L("inline_fields", q(";"), "field_decl"))
    g.rule("field_lines", [], L("field_lines", "field_line"))
    g.rule("field_line", [NL], L("field_decl", NL))
    g.rule("field_decl", L("ident_list", "type"), L("ident_list", "type", "tag"), L(q("*"), "IDENT"))
    g.rule("tag", ["STRING"], ["RAWSTRING"])
    g.rule("interface_type", L(q("interface"), q("{"), q("}")),
           L(q("interface"), q("{"), NL, "method_lines", q("}")))
    g.rule("method_lines", [], L("method_lines", "method_line"))
    g.rule("method_line", [NL], L("method_spec", NL))
    g.rule("method_spec", L("IDENT", "signature"), ["type_elem"])
    g.rule("type_elem", ["type_term"], L("type_elem", q("|"), "type_term"))
    g.rule("type_term", ["type"], L(q("~"), "type"))

    # ------------------------------------------------------------ statements
    g.rule("block", L(q("{"), "stmt_lines", "stmt_opt", q("}")))
    g.rule("stmt_lines", [], L("stmt_lines", "stmt_line"))
    g.rule("stmt_line", [NL], L("stmt", NL))
    g.rule("stmt_opt", [], ["stmt"])
    g.rule("stmt", ["simple_stmt"], ["decl"], ["return_stmt"], ["go_stmt"], ["defer_stmt"], ["if_stmt"],
           ["for_stmt"], ["switch_stmt"], ["select_stmt"], ["block"], ["branch_stmt"], ["sql_exec"],
           ["labeled_stmt"])
    g.rule("labeled_stmt", L("IDENT", q(":"), "stmt"))
    g.rule("simple_stmt", ["expr_list"], L("expr", q("<-"), "expr"), L("expr", q("++")), L("expr", q("--")),
           L("expr_list", "assign_op", "expr_list"), L("expr_list", q(":="), "expr_list"))
    g.rule("assign_op", *[[q(o)] for o in ["=", "+=", "-=", "*=", "/=", "%=", "&=", "|=", "^=", "<<=", ">>=",
                                            "&^="]])
    g.rule("return_stmt", [q("return")], L(q("return"), "expr_list"))
    g.rule("go_stmt", L(q("go"), "expr"))
    g.rule("defer_stmt", L(q("defer"), "expr"))
    g.rule("branch_stmt", [q("break")], [q("continue")], [q("fallthrough")], L(q("goto"), "IDENT"),
           L(q("break"), "IDENT"), L(q("continue"), "IDENT"))
    g.rule("if_stmt", L(q("if"), "if_header", "block", "else_part"))
    g.rule("if_header", ["expr"], L("simple_stmt", q(";"), "expr"))
    g.rule("else_part", [], L(q("else"), "if_stmt"), L(q("else"), "block"))
    g.rule("for_stmt", L(q("for"), "block"), L(q("for"), "expr", "block"), L(q("for"), "for_clause", "block"),
           L(q("for"), "range_clause", "block"))
    g.rule("for_clause", L("simple_opt", q(";"), "expr_opt", q(";"), "simple_opt"))
    g.rule("simple_opt", [], ["simple_stmt"])
    g.rule("expr_opt", [], ["expr"])
    g.rule("range_clause", L("expr_list", q(":="), q("range"), "expr"), L("expr_list", q("="), q("range"), "expr"),
           L(q("range"), "expr"))
    g.rule("switch_stmt", L(q("switch"), "switch_body"), L(q("switch"), "expr", "switch_body"),
           L(q("switch"), "simple_stmt", q(";"), "expr", "switch_body"))
    g.rule("switch_body", L(q("{"), "nl_lines", "case_clauses", q("}")))
    g.rule("case_clauses", [], L("case_clauses", "case_clause"))
    g.rule("case_clause", L("case_head", "stmt_lines"))
    g.rule("case_head", L(q("case"), "expr_list", q(":")), L(q("default"), q(":")))
    g.rule("select_stmt", L(q("select"), q("{"), "nl_lines", "comm_clauses", q("}")))
    g.rule("comm_clauses", [], L("comm_clauses", "comm_clause"))
    g.rule("comm_clause", L("comm_head", "stmt_lines"))
    g.rule("comm_head", L(q("case"), "simple_stmt", q(":")), L(q("default"), q(":")))

    # ------------------------------------------------------------ expressions
    g.rule("expr_list", ["expr"], L("expr_list", q(","), "expr"))
    g.rule("expr", ["or_expr"])
    g.rule("or_expr", ["and_expr"], L("or_expr", q("||"), "and_expr"))
    g.rule("and_expr", ["cmp_expr"], L("and_expr", q("&&"), "cmp_expr"))
    g.rule("cmp_expr", ["add_expr"], *[L("cmp_expr", q(o), "add_expr") for o in ["==", "!=", "<", "<=", ">", ">="]])
    g.rule("add_expr", ["mul_expr"], *[L("add_expr", q(o), "mul_expr") for o in ["+", "-", "|", "^"]])
    g.rule("mul_expr", ["unary_expr"], *[L("mul_expr", q(o), "unary_expr") for o in ["*", "/", "%", "<<", ">>", "&",
                                                                                  "&^"]])
    g.rule("unary_expr", ["primary"], *[L(q(o), "unary_expr") for o in ["+", "-", "!", "^", "*", "&", "<-"]])
    g.rule("primary", ["operand"], L("primary", q("."), "IDENT"), L("primary", q("["), "expr", q("]")),
           L("primary", q("["), "slice_bounds", q("]")), L("primary", q("."), q("("), "type", q(")")),
           L("primary", q("."), q("("), q("type"), q(")")), L("primary", q("("), "call_args", q(")")),
           L(q("["), q("]"), "type_name", q("("), "expr", q(")")))
    g.rule("slice_bounds", L("expr_opt", q(":"), "expr_opt"), L("expr_opt", q(":"), "expr", q(":"), "expr"))
    g.rule("call_args", [], ["expr_list"], L("expr_list", q(",")), L("expr_list", q("...")))
    g.rule("operand", ["literal"], ["IDENT"], L(q("("), "expr", q(")")), ["func_lit"], ["composite_lit"],
           ["sql_expr_atom"], ["alloc_call"])
    g.rule("alloc_call", L(q("make"), q("("), "type", q(")")), L(q("make"), q("("), "type", q(","), "expr_list", q(")")),
           L(q("new"), q("("), "type", q(")")))
    g.rule("literal", ["INT"], ["FLOAT"], ["STRING"], ["RAWSTRING"], ["SQ"], [q("nil")], [q("true")], [q("false")])
    g.rule("func_lit", L(q("func"), "signature", "block"))
    g.rule("composite_lit", L("literal_type", "lit_value"))
    g.rule("lit_value", L(q("{"), q("}")), L(q("{"), "elements", q("}")), L(q("{"), "elements", q(","), q("}")),
           L(q("{"), NL, "element_lines", q("}")))
    g.rule("elements", ["element"], L("elements", q(","), "element"))
    g.rule("element_lines", [], L("element_lines", "element", q(","), NL), L("element_lines", NL))
    g.rule("element", ["elem_value"], L("elem_value", q(":"), "elem_value"))
    g.rule("elem_value", ["expr"], ["lit_value"])

    # ------------------------------------------------------------ embedded SQL
    g.rule("sql_expr_atom", L(q("sql"), q("("), "sql_stmt", q(")")))
    g.rule("sql_exec", L(q("sql"), q("{"), "nl_lines", "sql_script", q("}")))
    g.rule("sql_script", [], L("sql_script", "sql_stmt", q(";"), "nl_lines"))
    g.rule("sql_stmt", ["query"], ["insert_stmt"], ["update_stmt"], ["delete_stmt"], ["create_stmt"],
           ["drop_stmt"], ["alter_stmt"], ["txn_stmt"], ["merge_stmt"], ["grant_stmt"], ["explain_stmt"],
           ["copy_stmt"], ["config_stmt"], ["prepare_stmt"], ["truncate_stmt"],
           L(q("REFRESH"), q("MATERIALIZED"), q("VIEW"), "table_name"),
           L(q("COMMENT"), q("ON"), "comment_target", q("IS"), "SQ"),
           L(q("VACUUM"), "vacuum_opts", "table_name"))
    g.rule("comment_target", L(q("TABLE"), "table_name"), L(q("COLUMN"), "IDENT", q("."), "IDENT"),
           L(q("VIEW"), "table_name"), L(q("INDEX"), "IDENT"))
    g.rule("vacuum_opts", [], [q("FULL")], [q("ANALYZE")], L(q("FULL"), q("ANALYZE")))
    g.rule("copy_stmt", L(q("COPY"), "table_name", "cols_opt", q("FROM"), "copy_src", "copy_opts"),
           L(q("COPY"), "table_name", "cols_opt", q("TO"), "copy_dst", "copy_opts"),
           L(q("COPY"), q("("), "query", q(")"), q("TO"), "copy_dst", "copy_opts"))
    g.rule("copy_src", ["SQ"], [q("STDIN")])
    g.rule("copy_dst", ["SQ"], [q("STDOUT")])
    g.rule("copy_opts", [], L(q("WITH"), q("("), "copy_opt_list", q(")")))
    g.rule("copy_opt_list", ["copy_opt"], L("copy_opt_list", q(","), "copy_opt"))
    g.rule("copy_opt", L(q("FORMAT"), q("CSV")), L(q("FORMAT"), q("TEXT")), [q("HEADER")],
           L(q("HEADER"), "bool_lit"), L(q("DELIMITER"), "SQ"))
    g.rule("bool_lit", [q("TRUE")], [q("FALSE")])
    g.rule("config_stmt", L(q("SET"), "IDENT", q("TO"), "config_value"), L(q("SET"), "IDENT", q("="), "config_value"),
           L(q("SHOW"), "IDENT"), L(q("RESET"), "IDENT"), L(q("RESET"), q("ALL")))
    g.rule("config_value", ["IDENT"], ["SQ"], ["INT"], [q("DEFAULT")])
    g.rule("prepare_stmt", L(q("PREPARE"), "IDENT", "prep_types", q("AS"), "sql_stmt"),
           L(q("EXECUTE"), "IDENT"), L(q("EXECUTE"), "IDENT", q("("), "sql_exprs", q(")")),
           L(q("DEALLOCATE"), "IDENT"), L(q("DEALLOCATE"), q("ALL")))
    g.rule("prep_types", [], L(q("("), "sql_type_list", q(")")))
    g.rule("sql_type_list", ["sql_type"], L("sql_type_list", q(","), "sql_type"))
    g.rule("truncate_stmt", L(q("TRUNCATE"), "table_name", "drop_mode"), L(q("TRUNCATE"), q("TABLE"), "table_name",
                                                                             "drop_mode"))
    g.rule("explain_stmt", L(q("EXPLAIN"), "query"), L(q("EXPLAIN"), q("ANALYZE"), "query"))
    g.rule("merge_stmt", L(q("MERGE"), q("INTO"), "table_name", "alias_opt", q("USING"), "table_primary", q("ON"),
                           "sql_expr", "merge_whens"))
    g.rule("merge_whens", ["merge_when"], L("merge_whens", "merge_when"))
    g.rule("merge_when", L(q("WHEN"), q("MATCHED"), "merge_and", q("THEN"), q("UPDATE"), q("SET"), "set_items"),
           L(q("WHEN"), q("MATCHED"), "merge_and", q("THEN"), q("DELETE")),
           L(q("WHEN"), q("NOT"), q("MATCHED"), "merge_and", q("THEN"), q("INSERT"), "cols_opt", q("VALUES"),
             "value_row"),
           L(q("WHEN"), q("NOT"), q("MATCHED"), "merge_and", q("THEN"), q("DO"), q("NOTHING")))
    g.rule("merge_and", [], L(q("AND"), "sql_expr"))
    g.rule("grant_stmt", L(q("GRANT"), "privileges", q("ON"), "grant_target", q("TO"), "grantees"),
           L(q("REVOKE"), "privileges", q("ON"), "grant_target", q("FROM"), "grantees"))
    g.rule("privileges", L(q("ALL"), q("PRIVILEGES")), [q("ALL")], ["privilege_list"])
    g.rule("privilege_list", ["privilege"], L("privilege_list", q(","), "privilege"))
    g.rule("privilege", [q("SELECT")], [q("INSERT")], [q("UPDATE")], [q("DELETE")], [q("EXECUTE")],
           [q("REFERENCES")], [q("TRIGGER")])
    g.rule("grant_target", ["table_name"], L(q("TABLE"), "table_name"), L(q("FUNCTION"), "table_name"))
    g.rule("grantees", ["grantee"], L("grantees", q(","), "grantee"))
    g.rule("grantee", ["IDENT"], [q("PUBLIC")])
    # queries
    g.rule("query", L("with_opt", "set_expr", "order_opt", "limit_opt", "lock_opt"))
    g.rule("lock_opt", [], L(q("FOR"), "lock_mode", "lock_wait"))
    g.rule("lock_mode", [q("UPDATE")], [q("SHARE")])
    g.rule("lock_wait", [], [q("NOWAIT")], L(q("SKIP"), q("LOCKED")))
    g.rule("with_opt", [], L(q("WITH"), "ctes"), L(q("WITH"), q("RECURSIVE"), "ctes"))
    g.rule("ctes", ["cte"], L("ctes", q(","), "cte"))
    g.rule("cte", L("IDENT", q("AS"), q("("), "query", q(")")),
           L("IDENT", q("("), "col_names", q(")"), q("AS"), q("("), "query", q(")")))
    g.rule("set_expr", ["select_core"], L("set_expr", "set_op", "select_core"))
    g.rule("set_op", [q("UNION")], L(q("UNION"), q("ALL")), [q("INTERSECT")], [q("EXCEPT")])
    g.rule("select_core", L(q("SELECT"), "distinct_opt", "select_list", "from_opt", "where_opt", "group_opt",
                            "having_opt", "window_opt"))
    g.rule("window_opt", [], L(q("WINDOW"), "window_defs"))
    g.rule("window_defs", ["window_def"], L("window_defs", q(","), "window_def"))
    g.rule("window_def", L("IDENT", q("AS"), q("("), "window_spec", q(")")))
    g.rule("window_spec", L("partition_opt", "order_opt", "frame_opt"))
    g.rule("distinct_opt", [], [q("DISTINCT")], [q("ALL")], L(q("DISTINCT"), q("ON"), q("("), "sql_exprs", q(")")))
    g.rule("select_list", ["select_items"], [q("*")])
    g.rule("select_items", ["select_item"], L("select_items", q(","), "select_item"))
    g.rule("select_item", ["sql_expr"], L("sql_expr", q("AS"), "IDENT"), L("sql_expr", "IDENT"),
           L("IDENT", q("."), q("*")))
    g.rule("from_opt", [], L(q("FROM"), "table_refs"))
    g.rule("table_refs", ["table_ref"], L("table_refs", q(","), "table_ref"))
    g.rule("table_ref", ["table_primary"], L("table_ref", "join_op", "table_primary", "join_cond"),
           L("table_ref", q("CROSS"), q("JOIN"), "table_primary"),
           L("table_ref", q("NATURAL"), q("JOIN"), "table_primary"),
           L("table_ref", q("NATURAL"), q("LEFT"), q("JOIN"), "table_primary"),
           L("table_ref", q("NATURAL"), q("RIGHT"), q("JOIN"), "table_primary"))
    g.rule("join_op", [q("JOIN")], L(q("INNER"), q("JOIN")), L(q("LEFT"), q("JOIN")),
           L(q("LEFT"), q("OUTER"), q("JOIN")), L(q("RIGHT"), q("JOIN")), L(q("RIGHT"), q("OUTER"), q("JOIN")),
           L(q("FULL"), q("JOIN")), L(q("FULL"), q("OUTER"), q("JOIN")))
    g.rule("join_cond", L(q("ON"), "sql_expr"), L(q("USING"), q("("), "col_names", q(")")))
    g.rule("table_primary", L("table_name", "alias_opt"), L(q("("), "query", q(")"), "alias_opt"),
           L(q("LATERAL"), q("("), "query", q(")"), "alias_opt"))
    g.rule("table_name", ["IDENT"], L("IDENT", q("."), "IDENT"))
    g.rule("alias_opt", [], ["IDENT"], L(q("AS"), "IDENT"), L(q("AS"), "IDENT", q("("), "col_names", q(")")))
    g.rule("col_names", ["IDENT"], L("col_names", q(","), "IDENT"))
    g.rule("where_opt", [], L(q("WHERE"), "sql_expr"))
    g.rule("group_opt", [], L(q("GROUP"), q("BY"), "group_items"))
    g.rule("group_items", ["group_item"], L("group_items", q(","), "group_item"))
    g.rule("group_item", ["sql_expr"], L(q("ROLLUP"), q("("), "sql_exprs", q(")")),
           L(q("CUBE"), q("("), "sql_exprs", q(")")), L(q("GROUPING"), q("SETS"), q("("), "grouping_sets", q(")")))
    g.rule("grouping_sets", ["grouping_set"], L("grouping_sets", q(","), "grouping_set"))
    g.rule("grouping_set", L(q("("), q(")")), L(q("("), "sql_exprs", q(")")))
    g.rule("having_opt", [], L(q("HAVING"), "sql_expr"))
    g.rule("order_opt", [], L(q("ORDER"), q("BY"), "order_items"))
    g.rule("order_items", ["order_item"], L("order_items", q(","), "order_item"))
    g.rule("order_item", L("sql_expr", "dir_opt", "nulls_opt"))
    g.rule("dir_opt", [], [q("ASC")], [q("DESC")])
    g.rule("nulls_opt", [], L(q("NULLS"), q("FIRST")), L(q("NULLS"), q("LAST")))
    g.rule("limit_opt", [], L(q("LIMIT"), "sql_add"), L(q("LIMIT"), q("ALL")), L(q("LIMIT"), "sql_add", q("OFFSET"), "sql_add"),
           L(q("OFFSET"), "sql_add", q("ROWS"), q("FETCH"), q("NEXT"), "sql_add", q("ROWS"), q("ONLY")))
    # data changes
    g.rule("insert_stmt", L("with_opt", q("INSERT"), q("INTO"), "table_name", "cols_opt", "insert_src", "conflict_opt",
                            "returning_opt"))
    g.rule("cols_opt", [], L(q("("), "col_names", q(")")))
    g.rule("insert_src", L(q("VALUES"), "value_rows"), ["query"], L(q("DEFAULT"), q("VALUES")))
    g.rule("value_rows", ["value_row"], L("value_rows", q(","), "value_row"))
    g.rule("value_row", L(q("("), "sql_exprs", q(")")))
    g.rule("conflict_opt", [], L(q("ON"), q("CONFLICT"), "cols_opt", q("DO"), q("NOTHING")),
           L(q("ON"), q("CONFLICT"), "cols_opt", q("DO"), q("UPDATE"), q("SET"), "set_items", "where_opt"))
    g.rule("returning_opt", [], L(q("RETURNING"), "select_list"))
    g.rule("update_stmt", L("with_opt", q("UPDATE"), "table_name", "alias_opt", q("SET"), "set_items", "from_opt", "where_opt",
                            "returning_opt"))
    g.rule("set_items", ["set_item"], L("set_items", q(","), "set_item"))
    g.rule("set_item", L("IDENT", q("="), "sql_expr"), L("IDENT", q("="), q("DEFAULT")))
    g.rule("delete_stmt", L("with_opt", q("DELETE"), q("FROM"), "table_name", "alias_opt", "using_opt", "where_opt",
                            "returning_opt"))
    g.rule("using_opt", [], L(q("USING"), "table_refs"))
    # definitions
    g.rule("create_stmt", L(q("CREATE"), "temp_opt", q("TABLE"), "if_not_exists", "table_name", q("("),
                            "table_elems", q(")")),
           L(q("CREATE"), "unique_opt", q("INDEX"), "if_not_exists", "IDENT", q("ON"), "table_name", q("("),
             "order_items", q(")"), "where_opt"),
           L(q("CREATE"), q("VIEW"), "table_name", "cols_opt", q("AS"), "query"),
           L(q("CREATE"), q("SCHEMA"), "if_not_exists", "IDENT"),
           L(q("CREATE"), q("TYPE"), "table_name", q("AS"), q("ENUM"), q("("), "enum_labels", q(")")),
           L(q("CREATE"), "temp_opt", q("TABLE"), "if_not_exists", "table_name", "cols_opt", q("AS"), "query"),
           L(q("CREATE"), q("MATERIALIZED"), q("VIEW"), "if_not_exists", "table_name", q("AS"), "query", "with_data"),
           L(q("CREATE"), q("FUNCTION"), "table_name", q("("), "func_params", q(")"), q("RETURNS"), "func_ret",
             q("AS"), "SQ", q("LANGUAGE"), "IDENT", "volatility"),
           L(q("CREATE"), q("SEQUENCE"), "if_not_exists", "table_name", "seq_opts"),
           L(q("CREATE"), q("TRIGGER"), "IDENT", "trigger_time", "trigger_events", q("ON"), "table_name",
             q("FOR"), q("EACH"), q("ROW"), "trigger_when", q("EXECUTE"), q("FUNCTION"), "IDENT", q("("), q(")")))
    g.rule("trigger_time", [q("BEFORE")], [q("AFTER")])
    g.rule("func_params", [], ["func_param_list"])
    g.rule("func_param_list", ["func_param"], L("func_param_list", q(","), "func_param"))
    g.rule("func_param", ["sql_type"], L("IDENT", "sql_type"))
    g.rule("func_ret", ["sql_type"], L(q("SETOF"), "sql_type"), L(q("TABLE"), q("("), "func_param_list", q(")")))
    g.rule("volatility", [], [q("IMMUTABLE")], [q("STABLE")], [q("VOLATILE")])
    g.rule("seq_opts", [], L("seq_opts", q("INCREMENT"), q("BY"), "INT"), L("seq_opts", q("START"), q("WITH"), "INT"))
    g.rule("trigger_events", ["trigger_event"], L("trigger_events", q("OR"), "trigger_event"))
    g.rule("trigger_event", [q("INSERT")], [q("UPDATE")], [q("DELETE")], L(q("UPDATE"), q("OF"), "col_names"))
    g.rule("trigger_when", [], L(q("WHEN"), q("("), "sql_expr", q(")")))
    g.rule("temp_opt", [], [q("TEMPORARY")])
    g.rule("enum_labels", ["SQ"], L("enum_labels", q(","), "SQ"))
    g.rule("with_data", [], L(q("WITH"), q("DATA")), L(q("WITH"), q("NO"), q("DATA")))
    g.rule("unique_opt", [], [q("UNIQUE")])
    g.rule("if_not_exists", [], L(q("IF"), q("NOT"), q("EXISTS")))
    g.rule("if_exists", [], L(q("IF"), q("EXISTS")))
    g.rule("table_elems", ["table_elem"], L("table_elems", q(","), "table_elem"))
    g.rule("table_elem", ["column_def"], ["table_constraint"])
    g.rule("column_def", L("IDENT", "sql_type", "col_constraints"))
    g.rule("col_constraints", [], L("col_constraints", "col_constraint"))
    g.rule("col_constraint", L(q("NOT"), q("NULL")), [q("NULL")], L(q("PRIMARY"), q("KEY")), [q("UNIQUE")],
           L(q("DEFAULT"), "sql_primary"), L(q("REFERENCES"), "table_name", "cols_opt"),
           L(q("CHECK"), q("("), "sql_expr", q(")")), L(q("CONSTRAINT"), "IDENT"))
    g.rule("table_constraint", L("constraint_name", q("PRIMARY"), q("KEY"), q("("), "col_names", q(")")),
           L("constraint_name", q("UNIQUE"), q("("), "col_names", q(")")),
           L("constraint_name", q("FOREIGN"), q("KEY"), q("("), "col_names", q(")"), q("REFERENCES"), "table_name",
             "cols_opt"),
           L("constraint_name", q("CHECK"), q("("), "sql_expr", q(")")))
    g.rule("constraint_name", [], L(q("CONSTRAINT"), "IDENT"))
    g.rule("sql_type", [q("INTEGER")], [q("BIGINT")], [q("SMALLINT")], [q("TEXT")], [q("BOOLEAN")], [q("REAL")],
           [q("DATE")], [q("TIME")], [q("TIMESTAMP")], [q("INTERVAL")], [q("BLOB")], [q("SERIAL")],
           L(q("DOUBLE"), q("PRECISION")), L(q("VARCHAR"), q("("), "INT", q(")")), L(q("CHAR"), q("("), "INT", q(")")),
           [q("NUMERIC")], L(q("NUMERIC"), q("("), "INT", q(")")), L(q("NUMERIC"), q("("), "INT", q(","), "INT", q(")")),
           L(q("DECIMAL"), q("("), "INT", q(","), "INT", q(")")))
    g.rule("drop_stmt", L(q("DROP"), "drop_kind", "if_exists", "table_name", "drop_mode"))
    g.rule("drop_kind", [q("TABLE")], [q("INDEX")], [q("VIEW")], [q("SCHEMA")], [q("SEQUENCE")],
           [q("TRIGGER")])
    g.rule("drop_mode", [], [q("CASCADE")], [q("RESTRICT")])
    g.rule("alter_stmt", L(q("ALTER"), q("TABLE"), "table_name", "alter_action"))
    g.rule("alter_action", L(q("ADD"), "column_def"), L(q("ADD"), q("COLUMN"), "column_def"),
           L(q("ADD"), "table_constraint"), L(q("DROP"), q("COLUMN"), "IDENT"), L(q("RENAME"), q("TO"), "IDENT"),
           L(q("RENAME"), q("COLUMN"), "IDENT", q("TO"), "IDENT"),
           L(q("ALTER"), q("COLUMN"), "IDENT", q("SET"), q("DEFAULT"), "sql_primary"),
           L(q("ALTER"), q("COLUMN"), "IDENT", q("DROP"), q("DEFAULT")),
           L(q("ALTER"), q("COLUMN"), "IDENT", q("SET"), q("NOT"), q("NULL")),
           L(q("ALTER"), q("COLUMN"), "IDENT", q("DROP"), q("NOT"), q("NULL")),
           L(q("ALTER"), q("COLUMN"), "IDENT", q("TYPE"), "sql_type"))
    g.rule("txn_stmt", [q("BEGIN")], L(q("BEGIN"), q("TRANSACTION")), [q("COMMIT")], [q("ROLLBACK")])
    # SQL expressions: OR < AND < NOT < predicates < || < + - < * / % < unary
    g.rule("sql_exprs", ["sql_expr"], L("sql_exprs", q(","), "sql_expr"))
    g.rule("sql_expr", ["sql_or"])
    g.rule("sql_or", ["sql_and"], L("sql_or", q("OR"), "sql_and"))
    g.rule("sql_and", ["sql_not"], L("sql_and", q("AND"), "sql_not"))
    g.rule("sql_not", ["sql_pred"], L(q("NOT"), "sql_not"))
    g.rule("sql_pred", ["sql_cat"], *[L("sql_cat", q(o), "sql_cat") for o in ["=", "<>", "!=", "<", "<=", ">", ">="]],
           L("sql_cat", q("IS"), q("NULL")), L("sql_cat", q("IS"), q("NOT"), q("NULL")),
           L("sql_cat", q("LIKE"), "sql_cat", "escape_opt"), L("sql_cat", q("NOT"), q("LIKE"), "sql_cat", "escape_opt"),
           L("sql_cat", q("SIMILAR"), q("TO"), "sql_cat"), L("sql_cat", q("NOT"), q("SIMILAR"), q("TO"), "sql_cat"),
           L("sql_cat", q("IS"), q("DISTINCT"), q("FROM"), "sql_cat"),
           L("sql_cat", q("IS"), q("NOT"), q("DISTINCT"), q("FROM"), "sql_cat"),
           L("sql_cat", q("IS"), "bool_lit"), L("sql_cat", q("IS"), q("NOT"), "bool_lit"),
           L("sql_cat", q("ILIKE"), "sql_cat"),
           L("sql_cat", q("BETWEEN"), "sql_add", q("AND"), "sql_add"),
           L("sql_cat", q("NOT"), q("BETWEEN"), "sql_add", q("AND"), "sql_add"),
           L("sql_cat", q("IN"), q("("), "in_items", q(")")), L("sql_cat", q("NOT"), q("IN"), q("("), "in_items", q(")")),
           L("sql_cat", "cmp_op", q("ANY"), q("("), "query", q(")")),
           L("sql_cat", "cmp_op", q("SOME"), q("("), "query", q(")")),
           L("sql_cat", "cmp_op", q("ALL"), q("("), "query", q(")")))
    g.rule("cmp_op", *[[q(o)] for o in ["=", "<>", "<", ">"]])
    g.rule("escape_opt", [], L(q("ESCAPE"), "SQ"))
    g.rule("in_items", ["sql_exprs"], ["query"])
    g.rule("sql_cat", ["sql_json"], L("sql_cat", q("||"), "sql_json"))
    g.rule("sql_json", ["sql_add"], *[L("sql_json", q(o), "sql_add") for o in ["->", "->>", "@>", "<@"]])
    g.rule("sql_add", ["sql_mul"], L("sql_add", q("+"), "sql_mul"), L("sql_add", q("-"), "sql_mul"))
    g.rule("sql_mul", ["sql_unary"], *[L("sql_mul", q(o), "sql_unary") for o in ["*", "/", "%"]])
    g.rule("sql_unary", ["sql_postfix"], L(q("-"), "sql_unary"), L(q("+"), "sql_unary"))
    g.rule("sql_postfix", ["sql_primary"], L("sql_postfix", q("::"), "sql_type"),
           L("sql_postfix", q("AT"), q("TIME"), q("ZONE"), "SQ"),
           L("sql_postfix", q("["), "sql_expr", q("]")))
    g.rule("sql_primary", ["sql_literal"], ["column_ref"], ["PARAM"], L(q("("), "sql_expr", q(")")),
           L(q("("), "query", q(")")), L(q("EXISTS"), q("("), "query", q(")")), ["case_expr"], ["func_call"],
           L(q("CAST"), q("("), "sql_expr", q("AS"), "sql_type", q(")")),
           L(q("EXTRACT"), q("("), "IDENT", q("FROM"), "sql_expr", q(")")),
           L(q("ARRAY"), q("["), q("]")), L(q("ARRAY"), q("["), "sql_exprs", q("]")), L(q("ARRAY"), q("("), "query", q(")")),
           ["string_func"], [q("CURRENT_DATE")], [q("CURRENT_TIME")], [q("CURRENT_TIMESTAMP")])
    g.rule("string_func", L(q("SUBSTRING"), q("("), "sql_expr", q("FROM"), "sql_expr", q(")")),
           L(q("SUBSTRING"), q("("), "sql_expr", q("FROM"), "sql_expr", q("FOR"), "sql_expr", q(")")),
           L(q("POSITION"), q("("), "sql_cat", q("IN"), "sql_cat", q(")")),
           L(q("TRIM"), q("("), "trim_spec", "sql_expr", q("FROM"), "sql_expr", q(")")),
           L(q("TRIM"), q("("), "sql_expr", q(")")),
           L(q("OVERLAY"), q("("), "sql_expr", q("PLACING"), "sql_expr", q("FROM"), "sql_expr", q(")")))
    g.rule("trim_spec", [q("BOTH")], [q("LEADING")], [q("TRAILING")])
    g.rule("sql_literal", ["INT"], ["FLOAT"], ["SQ"], [q("NULL")], [q("TRUE")], [q("FALSE")],
           L(q("INTERVAL"), "SQ"), L(q("DATE"), "SQ"), L(q("TIMESTAMP"), "SQ"))
    g.rule("column_ref", ["IDENT"], L("IDENT", q("."), "IDENT"))
    g.rule("case_expr", L(q("CASE"), "when_clauses", "else_opt", q("END")),
           L(q("CASE"), "sql_expr", "when_clauses", "else_opt", q("END")))
    g.rule("when_clauses", ["when_clause"], L("when_clauses", "when_clause"))
    g.rule("when_clause", L(q("WHEN"), "sql_expr", q("THEN"), "sql_expr"))
    g.rule("else_opt", [], L(q("ELSE"), "sql_expr"))
    g.rule("func_call", L("func_head", "within_opt", "filter_opt", "over_opt"))
    g.rule("within_opt", [], L(q("WITHIN"), q("GROUP"), q("("), q("ORDER"), q("BY"), "order_items", q(")")))
    g.rule("func_head", L("IDENT", q("("), q(")")), L("IDENT", q("("), "sql_exprs", q(")")),
           L("IDENT", q("("), "sql_exprs", q("ORDER"), q("BY"), "order_items", q(")")),
           L(q("COUNT"), q("("), q("*"), q(")")), L("agg_name", q("("), "sql_expr", q(")")),
           L("agg_name", q("("), q("DISTINCT"), "sql_expr", q(")")), L(q("COUNT"), q("("), "sql_expr", q(")")),
           L(q("COUNT"), q("("), q("DISTINCT"), "sql_expr", q(")")),
           L(q("COALESCE"), q("("), "sql_exprs", q(")")), L(q("NULLIF"), q("("), "sql_expr", q(","), "sql_expr", q(")")))
    g.rule("agg_name", [q("SUM")], [q("AVG")], [q("MIN")], [q("MAX")])
    g.rule("filter_opt", [], L(q("FILTER"), q("("), q("WHERE"), "sql_expr", q(")")))
    g.rule("over_opt", [], L(q("OVER"), q("("), "window_spec", q(")")), L(q("OVER"), "IDENT"))
    g.rule("partition_opt", [], L(q("PARTITION"), q("BY"), "sql_exprs"))
    g.rule("frame_opt", [], L("frame_unit", "frame_bound"),
           L("frame_unit", q("BETWEEN"), "frame_bound", q("AND"), "frame_bound"))
    g.rule("frame_unit", [q("ROWS")], [q("RANGE")])
    g.rule("frame_bound", L(q("UNBOUNDED"), q("PRECEDING")), L(q("UNBOUNDED"), q("FOLLOWING")),
           L(q("CURRENT"), q("ROW")), L("sql_add", q("PRECEDING")), L("sql_add", q("FOLLOWING")))
    return g.compile()


@functools.lru_cache(maxsize=None)
def grammar() -> GrammarTables:
    return gosql_grammar()


# ----------------------------------------------------------------- documents

IDENT_WORDS = ["x", "y", "i", "j", "n", "err", "ctx", "rows", "row", "db", "tx", "user", "users", "id", "name",
               "email", "orders", "order_id", "amount", "total", "price", "qty", "items", "item", "buf", "data",
               "key", "val", "cfg", "srv", "req", "resp", "log", "ch", "done", "mu", "wg", "result", "count",
               "created_at", "updated_at", "status", "customer", "product", "t", "u", "o", "p", "idx", "size",
               "handler", "Server", "Config", "Order", "User", "Store", "Repo", "Client", "fmt", "strings", "time",
               "sync", "http", "json", "Println", "Sprintf", "Now", "Query", "Exec", "Scan", "Next", "Close"]
_SPACELESS_AFTER = {"(", "[", "\n"}
_SPACELESS_BEFORE = {")", "]", ",", ";", "\n"}


class _Realiser:
    """Spellings of terminals: literals as written, regex terminals drawn
    from small pools (identifiers never equal a keyword)."""

    def __init__(self, g: GrammarTables, rng: np.random.Generator):
        self.g, self.r = g, rng
        self.names = g.terminal_names

    def text(self, t: int) -> str:
        name = self.names[t]
        if name.startswith('"'):
            return name[1:-1]
        r = self.r
        if name == "IDENT":
            w = IDENT_WORDS[int(r.integers(len(IDENT_WORDS)))]
            return w + str(int(r.integers(0, 10))) if r.random() < 0.15 else w
        if name == "INT":
            return str(int(r.integers(0, 1000)))
        if name == "FLOAT":
            return f"{int(r.integers(0, 100))}.{int(r.integers(0, 100))}"
        if name == "STRING":
            return '"' + IDENT_WORDS[int(r.integers(len(IDENT_WORDS)))] + '"'
        if name == "RAWSTRING":
            return "`" + IDENT_WORDS[int(r.integers(len(IDENT_WORDS)))] + "`"
        if name == "SQ":
            return "'" + IDENT_WORDS[int(r.integers(len(IDENT_WORDS)))] + "'"
        if name == "PARAM":
            return f"${int(r.integers(1, 9))}" if r.random() < 0.8 else "?"
        raise ValueError(f"no spelling for terminal {name}")


def _join(tokens: list[str]) -> str:
    out: list[str] = []
    prev = "\n"
    for t in tokens:
        if out and prev not in _SPACELESS_AFTER and t not in _SPACELESS_BEFORE:
            out.append(" ")
        out.append(t)
        prev = t
    return "".join(out)


# Relative weights of some productions, keyed by (left-hand side, first
# symbol of the body; "" for an empty body), so that random programs look
# like programs (functions with statements and queries) rather than lists
# of imports and blank lines; every other production weighs 1 (0.3 when
# empty).
_ALT_WEIGHTS = {
    ("top_item", '"\n"'): 0.2, ("top_item", "import_decl"): 0.4, ("top_item", "func_decl"): 3.0,
    ("top_item", "method_decl"): 1.5, ("top_item", "decl"): 0.8,
    ("nl_lines", "nl_lines"): 0.1, ("nl_plus", "nl_plus"): 0.1, ("stmt_line", '"\n"'): 0.15,
    ("stmt", "simple_stmt"): 4.0, ("stmt", "decl"): 0.5, ("stmt", "go_stmt"): 0.3, ("stmt", "defer_stmt"): 0.3,
    ("stmt", "select_stmt"): 0.2, ("stmt", "block"): 0.2, ("stmt", "branch_stmt"): 0.3, ("stmt", "labeled_stmt"): 0.1,
    ("stmt", "sql_exec"): 0.8, ("stmt", "if_stmt"): 1.5, ("stmt", "for_stmt"): 1.2, ("stmt", "switch_stmt"): 0.5,
    ("operand", "IDENT"): 4.0, ("operand", "literal"): 2.0, ("operand", "func_lit"): 0.15,
    ("operand", "composite_lit"): 0.4, ("operand", "sql_expr_atom"): 0.6, ("operand", "alloc_call"): 0.3,
    ("unary_expr", "primary"): 40.0, ("primary", "operand"): 30.0, ("or_expr", "and_expr"): 8.0,
    ("and_expr", "cmp_expr"): 8.0, ("cmp_expr", "add_expr"): 30.0, ("add_expr", "mul_expr"): 20.0,
    ("mul_expr", "unary_expr"): 40.0, ("type", "type_name"): 4.0, ("type_name", "IDENT"): 3.0,
    ("sql_or", "sql_and"): 8.0, ("sql_and", "sql_not"): 8.0, ("sql_not", "sql_pred"): 12.0,
    ("sql_pred", "sql_cat"): 12.0, ("sql_cat", "sql_json"): 12.0, ("sql_json", "sql_add"): 30.0,
    ("sql_add", "sql_mul"): 8.0, ("sql_mul", "sql_unary"): 15.0, ("sql_unary", "sql_postfix"): 20.0,
    ("sql_postfix", "sql_primary"): 20.0, ("sql_primary", "column_ref"): 8.0, ("sql_primary", "sql_literal"): 4.0,
    ("sql_primary", "PARAM"): 2.0, ("sql_stmt", "query"): 5.0, ("sql_stmt", "insert_stmt"): 1.5,
    ("sql_stmt", "update_stmt"): 1.5, ("sql_stmt", "delete_stmt"): 1.0,
}


class _Sentences:
    """Random sentences of the grammar: a leftmost derivation from the start
    symbol that picks productions at random until the derivation is deep or
    the output long, then finishes every open nonterminal by its shortest
    expansion (so every sentence is complete and in the language)."""

    def __init__(self, g: GrammarTables):
        self.g = g
        nt_names = g.nonterminal_names
        self.nt_index = {n: i for i, n in enumerate(nt_names)}
        self.term_index = {n: i for i, n in enumerate(g.terminal_names)}
        self.bodies: list[list[tuple[tuple[bool, int], ...]]] = [[] for _ in nt_names]
        for lhs, body in g.productions[1:]:
            enc = tuple((True, self.term_index[s]) if s in self.term_index else (False, self.nt_index[s]) for s in body)
            self.bodies[self.nt_index[lhs]].append(enc)
        # shortest expansion length of every nonterminal and production (fixpoint)
        INF = 10 ** 9
        cost = [INF] * len(nt_names)
        changed = True
        while changed:
            changed = False
            for a, alts in enumerate(self.bodies):
                for body in alts:
                    c = sum(1 if t else cost[x] for t, x in body)
                    if c < cost[a]:
                        cost[a], changed = c, True
        self.cost = cost
        self.short = [min(range(len(alts)), key=lambda k: sum(1 if t else cost[x] for t, x in alts[k]))
                      if alts else -1 for alts in self.bodies]
        self.weights = []
        names = g.terminal_names
        for a, alts in enumerate(self.bodies):
            w = []
            for body in alts:
                first = "" if not body else (names[body[0][1]] if body[0][0] else nt_names[body[0][1]])
                w.append(_ALT_WEIGHTS.get((nt_names[a], first), 0.3 if not body else 1.0))
            w = np.array(w, dtype=np.float64)
            self.weights.append(w / w.sum())

    def sentence(self, rng: np.random.Generator, start: str, max_depth: int, max_tokens: int) -> list[int]:
        out: list[int] = []
        stack: list[tuple[bool, int, int]] = [(False, self.nt_index[start], 0)]
        while stack:
            term, x, d = stack.pop()
            if term:
                out.append(x)
                continue
            alts = self.bodies[x]
            if d >= max_depth or len(out) + len(stack) >= max_tokens:
                body = alts[self.short[x]]
            else:
                # empty alternatives (ends of lists, absent options) a third
                # as likely as the others, so that lists are not cut short
                w = self.weights[x]
                body = alts[int(rng.choice(len(alts), p=w))]
            for t, y in reversed(body):
                stack.append((t, y, d + 1))
        return out


@functools.lru_cache(maxsize=None)
def _sentences() -> _Sentences:
    return _Sentences(grammar())


def program(rng: np.random.Generator) -> bytes:
    """A random complete program of the language (a random derivation of
    bounded depth and length)."""
    g = grammar()
    gen = _sentences()
    toks = gen.sentence(rng, "file", max_depth=int(rng.integers(18, 40)), max_tokens=int(rng.integers(150, 900)))
    real = _Realiser(g, rng)
    return _join([real.text(t) for t in toks]).encode()


# Openers that nest one level deeper and leave the prefix viable: the
# statement context of a block, an expression, or an SQL expression.
_BLOCK_OPENERS = ["if x > 0 {\n", "for i := range items {\n", "for {\n", "switch v {\ncase 1:\n",
                  "go func() {\n", "defer func() {\n", "select {\ncase v := <-ch:\n", "{\n",
                  "for i := 0; i < n; i++ {\n", "if err := f(); err != nil {\n", "else_marker"]
_EXPR_OPENERS = ["f(", "(", "a[", "[]int{", "map[string]int{\"k\": ", "g(x, ", "-(", "!(", "x + (", "y * (",
                 "h(a, b, ", "m[", "s.Get(", "[]string{\"a\", "]
_SQL_OPENERS = ["(", "x IN (SELECT id FROM t WHERE ", "COALESCE(", "NOT (", "a + (", "EXISTS (SELECT 1 FROM u WHERE ",
                "CASE WHEN ", "f(", "a = (", "(SELECT MAX(b) FROM v WHERE "]


def deep_program(rng: np.random.Generator, approx_chars: int = 6000) -> bytes:
    """A prefix that keeps nesting blocks, expressions and SQL subqueries and
    never closes them, interleaved with complete statements, so that the
    parser stack keeps growing (stack depths of several hundred)."""
    out = ["package main\n", "func run() {\n"]
    size = sum(len(s) for s in out)
    mode = "stmt"
    while size < approx_chars:
        r = rng.random()
        if mode == "stmt":
            if r < 0.45:
                s = _BLOCK_OPENERS[int(rng.integers(len(_BLOCK_OPENERS) - 1))]
            elif r < 0.6:
                s = ["x := 1\n", "n++\n", "err = db.Close()\n", "y = x * 2\n", "ch <- x\n"][int(rng.integers(5))]
            elif r < 0.8:
                s = "x = " + _EXPR_OPENERS[int(rng.integers(len(_EXPR_OPENERS)))]
                mode = "expr"
            else:
                s = "rows := sql(SELECT a, b FROM t WHERE " + _SQL_OPENERS[int(rng.integers(len(_SQL_OPENERS)))]
                mode = "sql"
        elif mode == "expr":
            if r < 0.85:
                s = _EXPR_OPENERS[int(rng.integers(len(_EXPR_OPENERS)))]
            else:
                s = "func() int {\n"
                mode = "stmt"
        else:
            s = _SQL_OPENERS[int(rng.integers(len(_SQL_OPENERS)))]
            if s == "CASE WHEN ":
                mode = "sqlcase"
        if mode == "sqlcase":
            s += "a > 1 THEN "
            mode = "sql"
        out.append(s)
        size += len(s)
    return "".join(out).encode()


def document(rng: np.random.Generator) -> bytes:
    """Most documents are complete random programs; one in four is a deeply
    nesting prefix (stack depths past 200)."""
    if rng.random() < 0.25:
        return deep_program(rng, approx_chars=int(rng.integers(800, 3000)))
    return program(rng)


def gosql_vocab(rng: np.random.Generator, V: int) -> Vocab:
    """Bytes + Zipf-length strings over identifiers, Go and SQL keywords,
    operators, punctuation runs and white space."""
    idents = [w.encode() for w in IDENT_WORDS] + [(w + "_" + v).encode() for w in IDENT_WORDS[:12]
                                                   for v in ("id", "at", "2")]
    kws = [k.encode() for k in GO_KEYWORDS + SQL_KEYWORDS] + [b" " + k.encode() for k in GO_KEYWORDS + SQL_KEYWORDS]
    ops = [o.encode() for o in GO_OPS + SQL_OPS] + [b" {\n", b"}\n", b"()", b"(\"", b"\")", b", ", b" := ", b" = ",
                                                     b" == ", b" != ", b"err != nil", b"sql(", b"$1", b"'", b'"']
    ws = [b" ", b"  ", b"\n", b"\n\t", b"\t", b"\t\t", b"\n\t\t"]
    digits = [bytes([c]) for c in b"0123456789"]
    pieces = idents + kws + ops + ws + digits
    weights = ([0.6] * len(idents) + [0.3] * len(kws) + [1.0] * len(ops) + [2.5] * len(ws) + [0.6] * len(digits))
    return piece_vocab(rng, V, pieces, weights, zipf_s=1.2, lo=2, hi=16)
